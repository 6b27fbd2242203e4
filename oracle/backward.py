"""Backward through time with the truncated surrogate (Sec. 2.2); oracle, test use only.

Notation (per layer, batch b implicit):
  eps_j[t]  gradient of the loss w.r.t. the layer's output spikes S_j[t]
            (for the readout: w.r.t. V_out[t]);
  G_j[t]    = eps_j[t] * dS_j[t]/dV_j[t], zero off the active set (Definition 2);
  delta_j[t] = sum_{k>t} alpha^{k-t-1} G_j[k]                    (Eq. (s_grad));
  dW_ij     = sum_t G_j[t] * trace_i[t]                          (Eq. (w_grad));
  eps_in_i[t] = sum_j W_ij delta_j[t]                            (Eq. (s_grad)).
The reset term is not differentiated (Sec. 2.2, after Eq. (w_grad)); the first
layer computes dW only.

Readings adopted: the trace in the sparse dW sum is sum_{k<t} alpha^{t-k-1}
S_i[k] (the printed S_i[t] inside the sum is an index slip); the summand of
delta is G_j[k] (not G_j[t]); the sparse spike gradient is eps_in_i[t] =
sum_j W_ij delta_j[t] where the presynaptic V_i[t] is active and 0 elsewhere.

Everything here is float64. Three variants compute the same numbers:
  O2 layer_backward         memoised delta recurrence + BLAS (production oracle)
  O1 layer_backward_literal the literal double sums, O(T^2) (tiny inputs)
  O3 layer_backward_events  Proposition 1 on event lists with the App. C
                            schedule, counting multiply-adds (tiny inputs)
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import numpy as np

from .active import active_mask, surrogate
from .loss import readout_grad

F64 = np.float64


def delta_recurrence(G: np.ndarray, alpha) -> np.ndarray:
    """delta[T-1] = 0 and delta[t] = alpha*delta[t+1] + G[t+1] (memoisation, App. B)."""
    a = float(alpha)
    D = np.zeros(G.shape, F64)
    for t in range(G.shape[0] - 2, -1, -1):
        D[t] = a * D[t + 1] + G[t + 1]
    return D


def layer_backward(G: np.ndarray, W: np.ndarray, trace: np.ndarray, alpha, grad_in: bool = True):
    """O2 for one layer: dW [N_in, N_out] and, if grad_in, eps_in [T, B, N_in] (dense).

    G [T, B, N_out] float64, W [N_in, N_out], trace [T, B, N_in].
    """
    T, B, n_out = G.shape
    n_in = trace.shape[2]
    G2 = np.asarray(G, F64).reshape(T * B, n_out)
    dW = np.asarray(trace, F64).reshape(T * B, n_in).T @ G2
    eps_in = None
    if grad_in:
        D = delta_recurrence(G, alpha)
        eps_in = (D.reshape(T * B, n_out) @ np.asarray(W, F64).T).reshape(T, B, n_in)
    return dW, eps_in


def csr_values(dense: np.ndarray, row_ptr: np.ndarray, col_idx: np.ndarray) -> np.ndarray:
    """Values of dense [T, B, N] at the CSR entries (rows r = t*B + b)."""
    T, B, N = dense.shape
    rows = np.repeat(np.arange(T * B), np.diff(row_ptr))
    return dense.reshape(T * B, N)[rows, col_idx]


def network_backward(fwd: dict, Ws, W_out, alphas, alpha_out, labels, mode: str,
                     theta, b_th, beta, absolute: bool = False, reg=None):
    """Gradients of the whole network (O2), top down.

    fwd: output of forward.network_forward. With absolute=True every weight is
    replaced by its absolute value and the loss gradient (p - y)/B by (p + y)/B,
    which yields the magnitude envelope used to state tolerances: every sum and
    difference of the chain taken with its terms in absolute value (traces, alpha
    and g are non-negative already).
    reg: optional list of [B, N_l] arrays, the derivative of an extra loss term
    w.r.t. the spike count of each neuron of LIF layer l (regularize.activity_grad);
    it joins eps[l] at every time step (in absolute value for the envelope).
    Returns dict with
      loss, dLda, readout (the readout_grad dict),
      dW_out, dW[l],
      eps[l]  dense gradient w.r.t. S of LIF layer l (index 0 = first layer),
      G[l], mask[l], g[l] (float64 surrogate at every entry).
    """
    L = len(Ws)
    ro = readout_grad(fwd["V_out"], labels, mode)
    G_out = ro["G_abs"] if absolute else ro["G"]
    Wo = np.abs(W_out) if absolute else W_out
    dW_out, eps = layer_backward(G_out, Wo, fwd["trace_out"], alpha_out, grad_in=True)
    dW = [None] * L
    eps_l = [None] * L
    Gs = [None] * L
    masks = [None] * L
    gs = [None] * L
    for l in range(L - 1, -1, -1):
        V = fwd["V"][l]
        if reg is not None and reg[l] is not None:
            c = np.asarray(reg[l], F64)[None]
            eps = eps + (np.abs(c) if absolute else c)
        mask = active_mask(V, theta, b_th)
        g = surrogate(V, theta, beta)
        G = eps * g * mask
        W = np.abs(Ws[l]) if absolute else Ws[l]
        eps_l[l] = eps
        Gs[l], masks[l], gs[l] = G, mask, g
        dW[l], eps = layer_backward(G, W, fwd["trace"][l], alphas[l], grad_in=l > 0)
    return {"loss": ro["loss"], "dLda": ro["dLda"], "readout": ro, "dW_out": dW_out, "dW": dW,
            "eps": eps_l, "G": Gs, "mask": masks, "g": gs}


# ------------------------------------------------------------------ O1

def layer_backward_literal(eps: np.ndarray, dSdV: np.ndarray, S_in: np.ndarray, W: np.ndarray, alpha):
    """O1: the double sums of Eqs. (w_grad) and (s_grad), recomputing every trace and
    delta from scratch (O(T^2)); the trace is built from the input spikes here."""
    T, B, n_out = eps.shape
    n_in = S_in.shape[2]
    a = float(alpha)
    G = np.asarray(eps, F64) * np.asarray(dSdV, F64)
    S = np.asarray(S_in != 0, F64)
    W = np.asarray(W, F64)
    dW = np.zeros((n_in, n_out))
    eps_in = np.zeros((T, B, n_in))
    for t in range(T):
        tr = np.zeros((B, n_in))
        for k in range(t):
            tr += a ** (t - k - 1) * S[k]
        dW += tr.T @ G[t]
        dl = np.zeros((B, n_out))
        for k in range(t + 1, T):
            dl += a ** (k - t - 1) * G[k]
        eps_in[t] = dl @ W.T
    return dW, eps_in


# ------------------------------------------------------------------ O3

def skip_delta(active: Dict[int, float], needed: Sequence[int], alpha, T: int):
    """Proposition 1 on events, in the App. C order.

    active: {t: G_j[t]} over the times t_j where dS_j/dV_j != 0;
    needed: the times t_i where delta_j is wanted.
    Starting from delta[T-1] = 0 it visits, from late to early, only the times t
    with t+1 in t_j (where delta gains a term) or t in t_i (where it is read), using
      delta[t] = alpha^n delta[t+n]            no active time in t+1..t+n,
      delta[t] = G[t+1] + alpha^n delta[t+n]   t+1 active, none in t+2..t+n,
    and stops after the earliest needed time.
    Returns ({t: delta[t] for t in needed}, visited times in order, #updates).
    """
    need = sorted(set(int(t) for t in needed))
    if not need:
        return {}, [], 0
    lo = need[0]
    a = float(alpha)
    events = sorted({int(t) - 1 for t in active if int(t) - 1 >= lo} | set(need), reverse=True)
    cur_t, cur = T - 1, 0.0
    out, visited = {}, []
    for t in events:
        n = cur_t - t
        val = a ** n * cur
        if (t + 1) in active:
            val += float(active[t + 1])
        cur_t, cur = t, val
        visited.append(t)
        if t in need:
            out[t] = val
    return out, visited, len(visited)


def layer_backward_events(G: np.ndarray, out_active: np.ndarray, trace: np.ndarray, W: np.ndarray, alpha,
                          in_active: Optional[np.ndarray] = None):
    """O3 for one layer: sparse dW and sparse eps_in with multiply-add counts.

    dW: each active output entry (t, b, j) adds G * trace[t, b, :] to column j.
    eps_in: for each (b, j) delta_j is evaluated by skip_delta at the times where
    some input neuron of sample b is active; each active input entry (t, b, i)
    then gets sum_j W_ij delta_j[t].
    Returns dW, eps_in (zero off in_active), counts dict.
    """
    T, B, n_out = G.shape
    n_in = trace.shape[2]
    W = np.asarray(W, F64)
    dW = np.zeros((n_in, n_out))
    madds_w = 0
    for t, b, j in zip(*np.nonzero(out_active)):
        dW[:, j] += G[t, b, j] * np.asarray(trace[t, b, :], F64)
        madds_w += n_in
    eps_in = np.zeros((T, B, n_in))
    madds_s = 0
    updates = 0
    if in_active is not None:
        for b in range(B):
            need = np.nonzero(in_active[:, b, :].any(axis=1))[0]
            delta_b = np.zeros((T, n_out))
            for j in range(n_out):
                act = {int(t): G[t, b, j] for t in np.nonzero(out_active[:, b, j])[0]}
                vals, _, n = skip_delta(act, need, alpha, T)
                updates += n
                for t, v in vals.items():
                    delta_b[t, j] = v
            for t, i in zip(*np.nonzero(in_active[:, b, :])):
                eps_in[t, b, i] = W[i] @ delta_b[t]
                madds_s += n_out
    return dW, eps_in, {"madds_w": madds_w, "madds_s": madds_s, "delta_updates": updates}
