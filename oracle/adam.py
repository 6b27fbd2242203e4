"""The Adam update (the optimiser of App. E's parameter table); oracle, test use only.

Adam as defined by Kingma and Ba (ICLR 2015, Algorithm 1), step k = 1, 2, ...:
    m <- beta1 m + (1 - beta1) g
    v <- beta2 v + (1 - beta2) g^2
    w <- w - lr * (m / (1 - beta1^k)) / (sqrt(v / (1 - beta2^k)) + eps)
with m = v = 0 before the first step. The appendix gives the learning rate and the
two betas; it does not give eps, which is taken as Adam's usual 1e-8.
Everything is float64.
"""
from __future__ import annotations

import numpy as np


def adam_update(w, g, m, v, step: int, lr: float, beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8):
    """One step; returns (w, m, v) as new float64 arrays."""
    if step < 1:
        raise ValueError("Adam steps count from 1")
    w = np.asarray(w, np.float64)
    g = np.asarray(g, np.float64)
    m = beta1 * np.asarray(m, np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, np.float64) + (1.0 - beta2) * g * g
    m_hat = m / (1.0 - beta1 ** step)
    v_hat = v / (1.0 - beta2 ** step)
    return w - lr * m_hat / (np.sqrt(v_hat) + eps), m, v
