"""Active set and truncated spike derivative (Definitions 1-2, Sec. 2.2); oracle, test use only.

* active iff |V - V_th| < B_th, strictly, decided in float32 (Eq. (active));
* dS/dV = g(V) on the active set and 0 elsewhere (Eq. (spike_derivative)), with
  g(V) = 1/(beta |V - V_th| + 1)^2 (Sec. 3; App. E "Surrogate gradient"),
  evaluated in float64 from the float32 V;
* the CSR lists the active entries of the [T, B, N] tensor row by row, rows
  r = t*B + b ascending, columns ascending inside a row.
"""
from __future__ import annotations

import numpy as np

F32 = np.float32


def active_mask(V: np.ndarray, theta, b_th) -> np.ndarray:
    """|V - theta| < b_th, every operand float32 (NaN is never active)."""
    V = np.asarray(V)
    if V.dtype == np.float64:
        return np.abs(V - float(theta)) < float(b_th)
    return np.abs(V - F32(theta)) < F32(b_th)


def surrogate(V: np.ndarray, theta, beta) -> np.ndarray:
    """g(V) = 1 / (beta |V - theta| + 1)^2 in float64."""
    d = np.abs(np.asarray(V, dtype=np.float64) - float(theta))
    return 1.0 / (float(beta) * d + 1.0) ** 2


def active_csr(V: np.ndarray, theta, b_th, beta):
    """CSR of the active set of V [T, B, N].

    Returns row_ptr int64 [T*B + 1], col_idx int64 [nnz], g float64 [nnz].
    """
    T, B, N = V.shape
    m = active_mask(V, theta, b_th).reshape(T * B, N)
    rows, cols = np.nonzero(m)
    row_ptr = np.zeros(T * B + 1, np.int64)
    np.cumsum(np.bincount(rows, minlength=T * B), out=row_ptr[1:])
    g = surrogate(V.reshape(T * B, N)[rows, cols], theta, beta)
    return row_ptr, cols.astype(np.int64), g
