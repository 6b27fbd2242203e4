"""One training step of the paper's network (App. E); oracle, test use only.

Loss = cross-entropy of the readout + the activity penalties of every LIF layer
(regularize.py); gradient = the truncated-surrogate BPTT of backward.py with the
penalties' gradient joining each layer's spike gradient; update = Adam (adam.py).
Setting b_th = inf gives the full-surrogate ("original") gradient the sparse one is
compared with (Sec. 3, App. H).
"""
from __future__ import annotations

import numpy as np

from .adam import adam_update
from .backward import network_backward
from .forward import network_forward
from .regularize import activity_grad, activity_penalty, spike_counts


def training_gradients(X, Ws, W_out, alphas, alpha_out, labels, mode, theta, b_th, beta, reg=None, fwd=None):
    """Loss parts and weight gradients at the given weights.

    reg = (lam_low, nu_low, lam_up, nu_up) or None. Returns the network_backward dict
    plus: ce (the cross-entropy), penalty (per layer, (1/B) sum_b R[b]), total,
    zeta (spike counts per layer), coef (per layer dR/dzeta), fwd.
    """
    if fwd is None:
        fwd = network_forward(X, Ws, W_out, alphas, alpha_out, np.float32(theta))
    zeta = [spike_counts(S) for S in fwd["S"]]
    if reg is not None:
        coef = [activity_grad(z, *reg) for z in zeta]
        pen = [float(activity_penalty(z, *reg).mean()) for z in zeta]
    else:
        coef = None
        pen = [0.0] * len(zeta)
    out = network_backward(fwd, Ws, W_out, alphas, alpha_out, labels, mode, theta, b_th, beta, reg=coef)
    out.update(ce=out["loss"], penalty=pen, total=out["loss"] + sum(pen), zeta=zeta, coef=coef, fwd=fwd)
    return out


def train_step(params, state, step, X, alphas, alpha_out, labels, mode, theta, b_th, beta, reg, lr,
               betas=(0.9, 0.999), eps=1e-8):
    """Gradients at params = [W_1, ..., W_L, W_out], then one Adam step per matrix.

    state = list of (m, v) pairs (zeros before the first step). Returns
    (new params, new state, the training_gradients dict).
    """
    Ws, W_out = params[:-1], params[-1]
    out = training_gradients(X, Ws, W_out, alphas, alpha_out, labels, mode, theta, b_th, beta, reg)
    grads = list(out["dW"]) + [out["dW_out"]]
    new_p, new_s = [], []
    for W, g, (m, v) in zip(params, grads, state):
        w2, m2, v2 = adam_update(W, g, m, v, step, lr, betas[0], betas[1], eps)
        new_p.append(w2)
        new_s.append((m2, v2))
    return new_p, new_s, out


def gradient_difference(dW_sparse, dW_full) -> dict:
    """Statistics of the difference between a sparse and a full-surrogate weight gradient (App. H).

    The appendix reports a maximum relative error between individual weights without
    stating the normalisation; three are given: the largest |difference| over the
    largest |full gradient|, the same per weight restricted to weights whose full
    gradient is at least 1% of the largest, and the relative Frobenius norm.
    Also the cosine similarity of the two gradients.
    """
    a = np.asarray(dW_sparse, np.float64).ravel()
    b = np.asarray(dW_full, np.float64).ravel()
    d = np.abs(a - b)
    scale = np.abs(b).max()
    big = np.abs(b) >= 0.01 * scale
    nb = np.linalg.norm(b)
    na = np.linalg.norm(a)
    return {
        "max_abs_over_max": float(d.max() / scale) if scale > 0 else 0.0,
        "max_rel_big": float((d[big] / np.abs(b[big])).max()) if big.any() else 0.0,
        "frobenius_rel": float(np.linalg.norm(a - b) / nb) if nb > 0 else 0.0,
        "cosine": float(a @ b / (na * nb)) if na > 0 and nb > 0 else 0.0,
    }
