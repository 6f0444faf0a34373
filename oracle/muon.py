"""Deflated polar factor (Muon) on the CPU, step by step.

Orientation follows the paper: a matrix A in R^{n x m} with n >= m. A wide
input is transposed first and its result transposed back, using
polar(M^T) = polar(M)^T (App. D, "Grouping").

Batched randomized SVD (Alg. 3), one matrix at a time (the batch is a loop):
    Y = A Omega,  Q = CholQR(Y)
    repeat J times:  Y = CholQR(A^T Q),  Q = CholQR(A Y)
    G = Q^T A,  G = U_G diag(s) V^T (thin SVD, s descending),  U = Q U_G,
    keep the leading r columns.
The sketch width is r' = min(m, k + p) for an absolute oversample p (the
paper's r + ceil(delta m), clipped at m).

Deflated polar factor (Alg. 1):
    gate (opt-in, tau > 0): fires if s_r < tau s_1; then
        k_eff = max{i : s_i > tau s_1}, else k_eff = 0.
    fixed rank (tau = 0): k_eff = k.
    k_eff > 0:  R = A - U_k diag(s_k) V_k^T,  nu = ||R||_F,
                X0 = R / nu + gamma^-1 U_k V_k^T
    k_eff = 0:  X0 = A / ||A||_F
    return N_L o ... o N_1 (X0).
Explicit restore (restore="explicit", the gamma -> infinity form of the
exact split polar(M) = U_k V_k^T + polar(R_k), eq:identities in Sec. 1):
    X0 = R / nu (no head term),  return U_k V_k^T + N_L o ... o N_1 (X0).
Degenerate scales (no epsilon is added, the paper has none): a zero nu or a
zero ||A||_F drops that term (a zero matrix maps to zero). Alg. 1 requires
k < rank(M); no other rule applies to nu.

Modes: "exact" (float64 throughout) and "bf16" (the bf16 contract). In the
bf16 contract the front end (randomized SVD, residual, start) is single
precision or better, as the paper runs its randomized SVD in single
precision (App. D, accuracy study); the oracle computes it in float64, so
it equals exact mode there. The filter then follows filters.ns_filter's
contract: every product takes bf16 operands, X0 and the iterates are stored
as bf16 hi plus an e4m3 residual (hi is the operand), and the output is
rounded to bf16.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .filters import ns_filter
from .linalg import cholqr
from .precision import rounding
from .rng import sketch



@dataclass
class MuonInfo:
    k_eff: list
    nu: list
    s: list
    rprime: int
    transposed: bool


def tall_view(m: np.ndarray) -> tuple[np.ndarray, bool]:
    m = np.asarray(m, dtype=np.float64)
    if m.shape[0] >= m.shape[1]:
        return m, False
    return m.T, True


def randomized_svd(a, r, rprime, power_iters, omega):
    """Alg. 3 for one tall matrix a (n x m). Returns U (n x r), s (r), V (m x r)."""
    q = cholqr(a @ omega)
    for _ in range(power_iters):
        y = cholqr(a.T @ q)
        q = cholqr(a @ y)
    g = q.T @ a
    ug, s, vt = np.linalg.svd(g, full_matrices=False)
    u = q @ ug
    return u[:, :r], s[:r], vt.T[:, :r]


def deflation_rank(s: np.ndarray, k: int, tau: float, r: int | None = None) -> int:
    """Number of deflated components: k in fixed-rank mode; with tau > 0 the
    gate of Alg. 1 over the first r estimated values (window, default k):
    when s_r < tau s_1 it deflates max{i : s_i > tau s_1} of them (fewer
    than r), capped at k; otherwise none."""
    if k == 0:
        return 0
    if tau <= 0.0:
        return k
    r = k if r is None else r
    if s[r - 1] < tau * s[0]:
        return min(k, int(np.count_nonzero(s[:r] > tau * s[0])))
    return 0


def deflated_init(a, u, s, v, k_eff, gamma, restore="padded"):
    """Start X0 of Alg. 1 (padded: the head enters at gamma^-1) or of the
    explicit restore (residual only), and the residual norm."""
    if k_eff == 0:
        nrm = float(np.linalg.norm(a))
        x0 = a / nrm if nrm > 0 else np.zeros_like(a)
        return x0, nrm
    uk, sk, vk = u[:, :k_eff], s[:k_eff], v[:, :k_eff]
    r = a - (uk * sk) @ vk.T
    nu = float(np.linalg.norm(r))
    x0 = r / nu if nu > 0 else np.zeros_like(r)
    if restore == "padded":
        x0 = x0 + (uk @ vk.T) / gamma
    return x0, nu


def msign_deflated(x, k, coeffs, *, oversample=8, power_iters=1, gamma=1.01,
                   tau=0.0, seed=0, mode="exact", sketches=None, restore="padded", window=None):
    """Deflated polar factor of every matrix of x [B, rows, cols] (float64
    values). coeffs: per-step table [L, 3]. Returns (out [B, rows, cols], info).
    sketches: optional list of Omega (m x r') overriding the generator.
    restore: "padded" (Alg. 1) or "explicit" (U_k V_k^T added after the
    filter; gamma is then unused). window: the gate's window r (Alg. 1;
    used only with tau > 0, default k): r triplets are estimated and the
    gate deflates k_eff = min(k, max{i : s_i > tau s_1}) of them when
    s_r < tau s_1."""
    if restore not in ("padded", "explicit"):
        raise ValueError(f"unknown restore {restore!r}")
    x = np.asarray(x, dtype=np.float64)
    outs, keff, nus, svals = [], [], [], []
    r = k if (tau <= 0.0 or not window) else int(window)
    rprime = 0
    transposed = False
    for b in range(x.shape[0]):
        a, transposed = tall_view(x[b])
        m = a.shape[1]
        if k > 0:
            rprime = min(m, r + oversample)
            omega = sketches[b] if sketches is not None else sketch(seed, b, m, rprime)
            u, s, v = randomized_svd(a, r, rprime, power_iters, omega)
            k_eff = deflation_rank(s, k, tau, r)
        else:
            u = s = v = None
            k_eff = 0
        x0, nu = deflated_init(a, u, s, v, k_eff, gamma, restore)
        xl = ns_filter(x0, coeffs, mode)
        if restore == "explicit" and k_eff > 0:
            xl = xl + u[:, :k_eff] @ v[:, :k_eff].T
        xl = rounding(mode)(xl)
        outs.append(xl.T if transposed else xl)
        keff.append(k_eff)
        nus.append(nu)
        svals.append(None if s is None else np.asarray(s))
    return np.stack(outs), MuonInfo(keff, nus, svals, rprime, transposed)


def msign(x, coeffs, *, mode="exact"):
    """Undeflated baseline: X0 = M / ||M||_F, then the filter (eq:muon_ns)."""
    out, _ = msign_deflated(x, 0, coeffs, mode=mode)
    return out


def polar_exact(m: np.ndarray) -> np.ndarray:
    """polar(M) = U V^T from a compact SVD (Sec. 1); batched over axis 0."""
    m = np.asarray(m, dtype=np.float64)
    u, _, vt = np.linalg.svd(m, full_matrices=False)
    return u @ vt
