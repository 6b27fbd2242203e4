"""Readout loss (App. E "Supervised and regularisation losses"); oracle, test use only.

Readings adopted:
* the readout is a LIF layer with infinite threshold (Sec. 3): no spikes, no
  reset, and the loss reads its membrane potential directly;
* logits a[b,c] = max_t V_out[t,b,c] for the latency, event and stress
  workloads and a[b,c] = sum_t V_out[t,b,c] for the audio (SHD-like) one, as
  App. E states per dataset; ties in the max go to the smallest t, and t = 0
  (V_out[0] = 0) takes part;
* the cross-entropy is the usual negative log-likelihood, mean over the batch
  (the appendix prints it without the minus sign);
* the activity regularisers of App. E live in regularize.py.
"""
from __future__ import annotations

import numpy as np


def readout_logits(V_out: np.ndarray, mode: str):
    """Logits [B, C] float64 and, for mode 'max', the first arg-max time [B, C]."""
    if mode == "max":
        tstar = np.argmax(V_out, axis=0)  # first maximal index
        return V_out.max(axis=0).astype(np.float64), tstar
    if mode == "sum":
        return V_out.astype(np.float64).sum(axis=0), None
    raise ValueError(mode)


def cross_entropy(a: np.ndarray, labels: np.ndarray, magnitude: bool = False):
    """Mean cross-entropy of softmax(a) and dL/da = (p - onehot) / B, float64.

    With magnitude=True the second result is (p + onehot) / B instead: the difference taken
    with its terms in absolute value, i.e. the scale on which rounding of p acts.
    """
    a = np.asarray(a, dtype=np.float64)
    B, C = a.shape
    z = a - a.max(axis=1, keepdims=True)
    p = np.exp(z)
    p /= p.sum(axis=1, keepdims=True)
    idx = (np.arange(B), np.asarray(labels))
    loss = -np.log(p[idx]).mean()
    d = p.copy()
    d[idx] += 1.0 if magnitude else -1.0
    return loss, d / B


def readout_grad(V_out: np.ndarray, labels: np.ndarray, mode: str):
    """Loss, dL/da, the dense dL/dV_out [T, B, C] and the readout's CSR.

    The CSR lists the entries of V_out that the loss reads (the arg-max entries
    for 'max', every entry for 'sum'), rows r = t*B + b, with eps = dL/da there;
    its derivative factor is 1 (the readout does not spike).
    Also returns G_abs, the same tensor built from (p + onehot)/B (see cross_entropy).
    Returns dict(loss, dLda, G, G_abs, row_ptr, col_idx, eps, tstar).
    """
    T, B, C = V_out.shape
    a, tstar = readout_logits(V_out, mode)
    loss, dLda = cross_entropy(a, labels)
    _, dLda_abs = cross_entropy(a, labels, magnitude=True)
    m = np.zeros((T, B, C), bool)
    if mode == "max":
        bb, cc = np.meshgrid(np.arange(B), np.arange(C), indexing="ij")
        m[tstar, bb, cc] = True
    else:
        m[:] = True
    G = np.where(m, dLda[None], 0.0)
    G_abs = np.where(m, dLda_abs[None], 0.0)
    rows, cols = np.nonzero(m.reshape(T * B, C))
    row_ptr = np.zeros(T * B + 1, np.int64)
    np.cumsum(np.bincount(rows, minlength=T * B), out=row_ptr[1:])
    eps = dLda[rows % B, cols]
    return {"loss": loss, "dLda": dLda, "G": G, "G_abs": G_abs, "row_ptr": row_ptr, "col_idx": cols.astype(np.int64), "eps": eps,
            "tstar": tstar}
