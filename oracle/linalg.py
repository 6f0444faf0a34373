"""CholeskyQR of tall panels (Alg. 3 and Alg. 2 orthonormalize with it).

One CholeskyQR pass on P (len x c), as the algorithms state:
    Gram = P^T P,   R^T R = Gram (Cholesky),   Q = P R^-1.
The Cholesky factor is computed column by column (left-looking). A pivot
that falls to or below the floor c u tr(Gram) (u = 2^-53) is replaced by the
floor: this never triggers for a panel of full numerical rank, and keeps a
rank-deficient panel finite. A zero panel (tr(Gram) = 0) maps to a zero Q.
In float64 the orthogonality error of one pass is about kappa(P)^2 u.
"""
from __future__ import annotations

import math

import numpy as np

UNIT_ROUNDOFF = 2.0 ** -53


def cholesky_upper(gram: np.ndarray, floor: float) -> np.ndarray:
    """Upper-triangular R with R^T R = gram, pivots floored at `floor`."""
    c = gram.shape[0]
    low = np.zeros_like(gram)
    for j in range(c):
        d = gram[j, j] - low[j, :j] @ low[j, :j]
        d = max(d, floor)
        low[j, j] = math.sqrt(d)
        low[j + 1:, j] = (gram[j + 1:, j] - low[j + 1:, :j] @ low[j, :j]) / low[j, j]
    return low.T


def cholqr(p: np.ndarray) -> np.ndarray:
    p = np.asarray(p, dtype=np.float64)
    c = p.shape[1]
    gram = p.T @ p
    tr = float(np.trace(gram))
    if tr == 0.0:
        return np.zeros_like(p)
    r = cholesky_upper(gram, c * UNIT_ROUNDOFF * tr)
    return np.linalg.solve(r.T, p.T).T                        # P R^-1
