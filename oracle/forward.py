"""LIF forward (Sec. 2.1, Eqs. (lif), (spike_fn), (lif_unrolled)); oracle, test use only.

Readings adopted where the paper is loose:
* time runs t = 0..T-1, V[0] = 0, so S_out[0] = 0; V[t+1] uses S_in[t] and
  S_out[t]; S_in[T-1] never enters V;
* the leak is +alpha (Eq. (lif); the appendix's "-alpha" is a sign slip);
* the reset subtracts V_th - V_r = 1 one step after the spike, undecayed, exactly
  as Eq. (lif) is written;
* a spike needs V > V_th strictly (Eq. (spike_fn));
* float32 throughout, each operation rounded on its own (no fused multiply-add),
  and the weighted input of a row is summed over its spiking inputs in
  ascending input index, starting from +0.0.
"""
from __future__ import annotations

import numpy as np

F32 = np.float32


def summed_inputs_loop(x: np.ndarray, W: np.ndarray) -> np.ndarray:
    """sum_i S_i W_ij for one time step, one element at a time (tiny inputs only).

    x: [B, N_in] bool, W: [N_in, N_out] float32 -> [B, N_out] float32.
    """
    B, n_in = x.shape
    n_out = W.shape[1]
    acc = np.zeros((B, n_out), F32)
    for b in range(B):
        for j in range(n_out):
            s = F32(0.0)
            for i in range(n_in):
                if x[b, i]:
                    s = F32(s + W[i, j])
            acc[b, j] = s
    return acc


def summed_inputs(x: np.ndarray, W: np.ndarray) -> np.ndarray:
    """sum_i S_i W_ij for one time step, same order as summed_inputs_loop.

    Each row adds its k-th spiking input (ascending i) in round k; a round adds
    one float32 row of W to each row that has a k-th spike, so every row sees
    ((0 + W[i1]) + W[i2]) + ... in its own ascending order.
    """
    B = x.shape[0]
    acc = np.zeros((B, W.shape[1]), F32)
    rows, cols = np.nonzero(x)
    if rows.size == 0:
        return acc
    counts = np.bincount(rows, minlength=B)
    first = np.concatenate(([0], np.cumsum(counts)[:-1]))
    rank = np.arange(rows.size) - first[rows]
    for k in range(int(counts.max())):
        sel = rank == k
        acc[rows[sel]] += W[cols[sel]]
    return acc


def lif_forward(X: np.ndarray, W: np.ndarray, alpha, theta):
    """One LIF layer over T steps.

    X: [T, B, N_in] spikes (nonzero = spike); W: [N_in, N_out] float32;
    alpha = exp(-dt/tau) and theta = V_th as float32; theta = +inf gives the
    non-spiking readout.
    Returns V [T, B, N_out] f32, S_out [T, B, N_out] u8 and the input trace
    [T, B, N_in] f32 with trace[0] = 0, trace[t+1] = alpha*trace[t] + S_in[t]
    (the filtered input of Eq. (lif_unrolled) that Eq. (w_grad) reuses).
    """
    W = np.asarray(W, dtype=F32)
    alpha = F32(alpha)
    theta = F32(theta)
    T, B, n_in = X.shape
    n_out = W.shape[1]
    V = np.zeros((T, B, n_out), F32)
    S = np.zeros((T, B, n_out), np.uint8)
    trace = np.zeros((T, B, n_in), F32)
    v = np.zeros((B, n_out), F32)
    tr = np.zeros((B, n_in), F32)
    for t in range(T):
        V[t] = v
        s = v > theta
        S[t] = s
        trace[t] = tr
        if t == T - 1:
            break
        x = X[t] != 0
        acc = summed_inputs(x, W)
        v = (alpha * v + acc) - s.astype(F32)
        tr = alpha * tr + x.astype(F32)
    return V, S, trace


def network_forward(X, Ws, W_out, alphas, alpha_out, theta=1.0):
    """L LIF layers then the infinite-threshold readout (Sec. 3).

    Returns a dict with per-layer lists V, S, trace (index 0 = first LIF layer)
    and V_out, trace_out for the readout.
    """
    Vs, Ss, trs = [], [], []
    x = X
    for W, a in zip(Ws, alphas):
        V, S, tr = lif_forward(x, W, a, theta)
        Vs.append(V)
        Ss.append(S)
        trs.append(tr)
        x = S
    V_out, _, tr_out = lif_forward(x, W_out, alpha_out, np.inf)
    return {"V": Vs, "S": Ss, "trace": trs, "V_out": V_out, "trace_out": tr_out}
