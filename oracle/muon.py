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
zero ||A||_F drops that term (a zero matrix maps to zero).
Residual floor (the degenerate case rank(A) <= k_eff): Sec. 2 notes that
inexact triplets leave components of R along the head directions and pads
the head at gamma^-1 against them; with exact triplets ||X0||_2 <= 1. When
nu is itself at the rounding level of the head, those components are not
small against nu and X0 can leave the filter's convergence interval. So a
residual with nu <= rho ||A||_F, where ||A||_F^2 = sum_{j < k_eff} s_j^2 +
nu^2 (U_k S_k V_k^T projects A on the head), is dropped like a zero one:
X0 = gamma^-1 U_k V_k^T (padded) or 0 (explicit). rho is the resolution
of the arithmetic that forms the head: 2^-8 for the bf16 contract (bf16
sketch operands), 2^-16 for the float32 kernels that "exact" mode serves
as the reference of.

Modes: "exact" (float64 throughout) and "bf16" (the bf16 contract: the sketch
products take bf16 operands Omega, Q and Y; X0 is formed wide, and X0 and the
iterates are stored as bf16 hi plus an e4m3 residual, hi being every filter
product's operand (filters.ns_filter); the output is rounded to bf16).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .filters import ns_filter
from .linalg import cholqr
from .precision import rounding
from .rng import sketch


RESIDUAL_FLOOR = {"exact": 2.0 ** -16, "bf16": 2.0 ** -8}


@dataclass
class MuonInfo:
    k_eff: list
    nu: list
    s: list
    rprime: int
    transposed: bool
    floored: list


def tall_view(m: np.ndarray) -> tuple[np.ndarray, bool]:
    m = np.asarray(m, dtype=np.float64)
    if m.shape[0] >= m.shape[1]:
        return m, False
    return m.T, True


def randomized_svd(a, r, rprime, power_iters, omega, mode="exact"):
    """Alg. 3 for one tall matrix a (n x m). Returns U (n x r), s (r), V (m x r)."""
    rd = rounding(mode)
    q = cholqr(a @ rd(omega))
    for _ in range(power_iters):
        y = cholqr(a.T @ rd(q))
        q = cholqr(a @ rd(y))
    g = rd(q).T @ a
    ug, s, vt = np.linalg.svd(g, full_matrices=False)
    u = q @ ug
    return u[:, :r], s[:r], vt.T[:, :r]


def deflation_rank(s: np.ndarray, k: int, tau: float) -> int:
    """Number of deflated components: k in fixed-rank mode, the gate of
    Alg. 1 on the k estimated values otherwise."""
    if k == 0:
        return 0
    if tau <= 0.0:
        return k
    if s[k - 1] < tau * s[0]:
        return int(np.count_nonzero(s[:k] > tau * s[0]))
    return 0


def deflated_init(a, u, s, v, k_eff, gamma, restore="padded", rho=0.0):
    """Start X0 of Alg. 1 (padded: the head enters at gamma^-1) or of the
    explicit restore (residual only), the residual norm, and whether the
    residual fell to the floor rho ||A||_F and was dropped."""
    if k_eff == 0:
        nrm = float(np.linalg.norm(a))
        x0 = a / nrm if nrm > 0 else np.zeros_like(a)
        return x0, nrm, False
    uk, sk, vk = u[:, :k_eff], s[:k_eff], v[:, :k_eff]
    r = a - (uk * sk) @ vk.T
    nu = float(np.linalg.norm(r))
    floored = nu <= rho * float(np.sqrt(np.sum(sk * sk) + nu * nu))
    x0 = r / nu if nu > 0 and not floored else np.zeros_like(r)
    if restore == "padded":
        x0 = x0 + (uk @ vk.T) / gamma
    return x0, nu, floored


def msign_deflated(x, k, coeffs, *, oversample=8, power_iters=1, gamma=1.01,
                   tau=0.0, seed=0, mode="exact", sketches=None, restore="padded", rho=None):
    """Deflated polar factor of every matrix of x [B, rows, cols] (float64
    values). coeffs: per-step table [L, 3]. Returns (out [B, rows, cols], info).
    sketches: optional list of Omega (m x r') overriding the generator.
    restore: "padded" (Alg. 1) or "explicit" (U_k V_k^T added after the
    filter; gamma is then unused). rho: residual floor (default
    RESIDUAL_FLOOR[mode]; 0 turns it off)."""
    if restore not in ("padded", "explicit"):
        raise ValueError(f"unknown restore {restore!r}")
    if rho is None:
        rho = RESIDUAL_FLOOR[mode]
    x = np.asarray(x, dtype=np.float64)
    outs, keff, nus, svals, floors = [], [], [], [], []
    rprime = 0
    transposed = False
    for b in range(x.shape[0]):
        a, transposed = tall_view(x[b])
        m = a.shape[1]
        if k > 0:
            rprime = min(m, k + oversample)
            omega = sketches[b] if sketches is not None else sketch(seed, b, m, rprime)
            u, s, v = randomized_svd(a, k, rprime, power_iters, omega, mode)
            k_eff = deflation_rank(s, k, tau)
        else:
            u = s = v = None
            k_eff = 0
        x0, nu, floored = deflated_init(a, u, s, v, k_eff, gamma, restore, rho)
        xl = ns_filter(x0, coeffs, mode)
        if restore == "explicit" and k_eff > 0:
            xl = xl + u[:, :k_eff] @ v[:, :k_eff].T
        xl = rounding(mode)(xl)
        outs.append(xl.T if transposed else xl)
        keff.append(k_eff)
        nus.append(nu)
        svals.append(None if s is None else np.asarray(s))
        floors.append(floored)
    return np.stack(outs), MuonInfo(keff, nus, svals, rprime, transposed, floors)


def msign(x, coeffs, *, mode="exact"):
    """Undeflated baseline: X0 = M / ||M||_F, then the filter (eq:muon_ns)."""
    out, _ = msign_deflated(x, 0, coeffs, mode=mode)
    return out


def polar_exact(m: np.ndarray) -> np.ndarray:
    """polar(M) = U V^T from a compact SVD (Sec. 1); batched over axis 0."""
    m = np.asarray(m, dtype=np.float64)
    u, _, vt = np.linalg.svd(m, full_matrices=False)
    return u @ vt
