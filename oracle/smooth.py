"""A smoothed-surrogate model for finite-difference checks; oracle, test use only.

Around a base point W0 with hard forward trajectory (Vbar, Sbar), define a model
M(W) in float64 in which
  * each LIF layer runs V[t+1] = alpha V[t] + sum_i X_i[t] W_ij - Sbar_j[t]
    (the reset uses the frozen base spikes: it is not differentiated, Sec. 2.2);
  * each LIF layer emits X_j[t] = Sbar_j[t] + s(V_j[t]) - s(Vbar_j[t]) with
    s(v) = sign(v - theta) (1/beta) (1 - 1/(1 + beta min(|v - theta|, B_th))),
    so that s'(v) = g(v) inside the band |v - theta| < B_th and 0 outside
    (Definitions 1-2, with g of App. E);
  * the readout and loss are those of loss.py.
At W0 the model reproduces the hard forward exactly, and its exact gradient is
the truncated-surrogate BPTT gradient of Eqs. (w_grad), (s_grad). Central
differences of M therefore check backward.network_backward independently of
its algebra.
"""
from __future__ import annotations

import numpy as np

from .loss import cross_entropy
from .regularize import activity_penalty


def hard_forward64(X, Ws, W_out, alphas, alpha_out, theta=1.0):
    """The LIF network of forward.network_forward in float64 (matrix products, any order)."""
    x = np.asarray(X != 0, np.float64)
    T = x.shape[0]
    Vs, Ss, trs = [], [], []
    layers = [(W, a, theta) for W, a in zip(Ws, alphas)] + [(W_out, alpha_out, np.inf)]
    for W, a, th in layers:
        W = np.asarray(W, np.float64)
        a = float(a)
        B = x.shape[1]
        V = np.zeros((T, B, W.shape[1]))
        S = np.zeros_like(V)
        tr = np.zeros_like(x)
        for t in range(T - 1):
            S[t] = V[t] > th
            V[t + 1] = a * V[t] + x[t] @ W - S[t]
            tr[t + 1] = a * tr[t] + x[t]
        S[T - 1] = V[T - 1] > th
        Vs.append(V)
        Ss.append(S)
        trs.append(tr)
        x = S
    return {"V": Vs[:-1], "S": Ss[:-1], "trace": trs[:-1], "V_out": Vs[-1], "trace_out": trs[-1]}


def s_tilde(v, theta, b_th, beta):
    d = v - theta
    a = np.minimum(np.abs(d), b_th)
    return np.sign(d) * (1.0 / beta) * (1.0 - 1.0 / (1.0 + beta * a))


def smoothed_losses(X, Ws, W_out, alphas, alpha_out, labels, mode, theta, b_th, beta, base, tstar=None,
                    reg=None):
    """Loss of M for a stack of P weight sets.

    Ws[l] and W_out may be [N_in, N_out] or [P, N_in, N_out]; base is the
    hard_forward64 dict at W0. For mode 'max' the arg-max times tstar [B, C] of
    the base point are used (the max is smooth where the arg-max is unique).
    reg = (lam_low, nu_low, lam_up, nu_up) adds the activity penalties of every LIF
    layer, evaluated on the smoothed counts sum_t X_j[t] (a continuous function of W
    that equals the spike count at W0).
    Returns losses [P].
    """
    x = np.asarray(X != 0, np.float64)[None]  # [1, T, B, N]
    T = x.shape[1]
    extra = 0.0
    layers = list(zip(Ws, alphas))
    for l, (W, a) in enumerate(layers):
        W = np.asarray(W, np.float64)
        if W.ndim == 2:
            W = W[None]
        a = float(a)
        Sb = base["S"][l][None]
        Vb = base["V"][l][None]
        P = max(W.shape[0], x.shape[0])
        V = np.zeros((P, T, x.shape[2], W.shape[2]))
        for t in range(T - 1):
            V[:, t + 1] = a * V[:, t] + np.matmul(x[:, t], W) - Sb[:, t]
        x = Sb + s_tilde(V, theta, b_th, beta) - s_tilde(Vb, theta, b_th, beta)
        if reg is not None:
            zeta = x.sum(axis=1)  # [P, B, N]
            extra = extra + activity_penalty(zeta, *reg).mean(axis=-1)
    Wo = np.asarray(W_out, np.float64)
    if Wo.ndim == 2:
        Wo = Wo[None]
    P = max(Wo.shape[0], x.shape[0])
    Vo = np.zeros((P, T, x.shape[2], Wo.shape[2]))
    ao = float(alpha_out)
    for t in range(T - 1):
        Vo[:, t + 1] = ao * Vo[:, t] + np.matmul(x[:, t], Wo)
    if mode == "max":
        B, C = tstar.shape
        bb, cc = np.meshgrid(np.arange(B), np.arange(C), indexing="ij")
        logits = Vo[:, tstar, bb, cc]
    else:
        logits = Vo.sum(axis=1)
    ce = np.array([cross_entropy(logits[p], labels)[0] for p in range(P)])
    return ce + extra
