"""CholeskyQR of tall panels (Alg. 3 and Alg. 2 orthonormalize with it).

One CholeskyQR pass on P (len x c):  Gram = P^T P,  R^T R = Gram + sigma I,
Q = P R^-1.  The tiny shift sigma = 11 (len c + c (c + 1)) u tr(Gram) with
u = 2^-53 is the one of shifted CholeskyQR (Fukaya, Kannan, Nakatsukasa,
Yamamoto, Yanagisawa, SIAM J. Sci. Comput. 2020) for a float64 Gram; it keeps
the factorization defined when the panel is rank deficient and changes a
well-conditioned result only at the 1e-10 level. A zero panel (tr(Gram) = 0)
maps to a zero Q. The paper applies "CholeskyQR" once; here it is applied twice
(CholeskyQR2), which restores orthogonality to working precision for the
condition numbers the sketches reach.
"""
from __future__ import annotations

import numpy as np

UNIT_ROUNDOFF = 2.0 ** -53


def cholqr_once(p: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    p = np.asarray(p, dtype=np.float64)
    n, c = p.shape
    gram = p.T @ p
    tr = float(np.trace(gram))
    if tr == 0.0:
        return np.zeros_like(p), np.zeros((c, c))
    sigma = 11.0 * (n * c + c * (c + 1)) * UNIT_ROUNDOFF * tr
    r = np.linalg.cholesky(gram + sigma * np.eye(c)).T       # upper, R^T R
    q = np.linalg.solve(r.T, p.T).T                           # P R^-1
    return q, r


def cholqr2(p: np.ndarray) -> np.ndarray:
    q, _ = cholqr_once(p)
    q, _ = cholqr_once(q)
    return q
