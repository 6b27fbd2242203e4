"""Activity regularisers of App. E ("Supervised and regularisation losses"); oracle, test use only.

For every LIF layer l with N neurons and spike counts zeta[b, i] = sum_t S_i[t] of
sample b, the appendix adds two per-sample penalties to the cross-entropy: a lower
activity term on each neuron's count and an upper activity term on the layer's mean
count, averaged over the batch.

Readings adopted:
* Signs: the appendix prints both penalties with a leading minus, and its
  cross-entropy without one, i.e. as quantities to be maximised. The loss minimised
  here is the negation: per sample
      R_low[b] = (lam_low / N) sum_i max(0, nu_low - zeta[b, i])^2
      R_up[b]  =  lam_up max(0, (1/N) sum_i zeta[b, i] - nu_up)
  (both >= 0), and the total is CE + (1/B) sum_l sum_b (R_low[b] + R_up[b]) over
  every LIF layer (the readout does not spike and has no such term).
* The slope of max(0, x) at x = 0 is taken as 0.
* The count is a plain sum over time, so dR/dS_i[t] = dR/dzeta_i at every t; that
  gradient then reaches V through the (truncated) surrogate exactly like the
  gradient from the layer above.

Everything is float64; zeta may be real-valued (the smoothed model of smooth.py
feeds continuous counts).
"""
from __future__ import annotations

import numpy as np


def spike_counts(S: np.ndarray) -> np.ndarray:
    """zeta [B, N] int64: spikes of each neuron per sample over all T steps (any nonzero byte)."""
    return (np.asarray(S) != 0).sum(axis=0).astype(np.int64)


def activity_penalty(zeta, lam_low, nu_low, lam_up, nu_up) -> np.ndarray:
    """Per-sample penalty R_low[b] + R_up[b], float64 [B]."""
    z = np.asarray(zeta, np.float64)
    N = z.shape[-1]
    low = (lam_low / N) * (np.maximum(0.0, nu_low - z) ** 2).sum(axis=-1)
    up = lam_up * np.maximum(0.0, z.mean(axis=-1) - nu_up)
    return low + up


def activity_grad(zeta, lam_low, nu_low, lam_up, nu_up) -> np.ndarray:
    """coef [B, N] float64: derivative of (1/B) sum_b (R_low[b] + R_up[b]) w.r.t. zeta[b, i]."""
    z = np.asarray(zeta, np.float64)
    B, N = z.shape
    low = -2.0 * (lam_low / N) * np.maximum(0.0, nu_low - z)
    up = np.where(z.mean(axis=1, keepdims=True) > nu_up, lam_up / N, 0.0)
    return (low + up) / B
