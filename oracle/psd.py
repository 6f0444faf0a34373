"""Deflated PSD projection on the CPU, step by step.

Lanczos scale estimate (App. E.1, "Normalization scale"): 20 Lanczos steps on
B = R^2 (applied as R (R x), never formed) from a random start; with (rho, v)
the largest Ritz pair, theta = sqrt(rho + ||B v - rho v||_2). Readings where
the paper is silent: the start is the seeded Gaussian of rng.lanczos_start,
normalized; every new Lanczos vector is reorthogonalized against all previous
ones (two classical Gram-Schmidt passes); the run stops early when the new
off-diagonal is exactly zero; the step count is capped at n.

Deflated projection (Alg. 2), one call:
    (J - 1) pre-steps  V = CholQR(Z V)
    Zt = Z V;  V^T Zt = E diag(lam) E^T;  U = V E
    order the Ritz pairs by |lam| descending (ties: larger lam first, then
    the original index)
    gate (opt-in, tau > 0): fires if s_r < tau s_1 with s = sorted |lam| and
        r the window; then I = {i : |lam_i| > tau s_1}, else I is empty.
    fixed rank (tau = 0): I = all K pairs.
    I non-empty:
        R = Z - sum_I lam_i u_i u_i^T,  theta = Lanczos estimate of ||R||_2
        X0 = R / theta + gamma^-1 sum_I sign(lam_i) u_i u_i^T
        P = 1/2 R (I + g(X0)) + sum_{I, lam_i > 0} lam_i u_i u_i^T
    I empty (eq:baseline_projection):
        theta = Lanczos estimate of ||Z||_2,  X0 = Z / theta,
        P = 1/2 Z (I + g(X0))
    P = 1/2 (P + P^T)  (Sec. 2.3),   V_next = CholQR(Zt).
g is the Newton-Schulz composition (filters.ns_filter) with a per-step
coefficient table; the default is the cubic Bjorck-Bowie map (3/2, -1/2).
A zero theta drops the R / theta term.
scale "frobenius" replaces the Lanczos estimate by theta = ||R||_F (or
||Z||_F undeflated), an upper bound on ||R||_2 that needs no iteration: the
residual is then Frobenius-normalized, as Alg. 1 normalizes its residual.
fp16 mode (the fp16 projection of the paper's SDP runs): every product of the
filter stage takes fp16 operands, the restore product R g included, whose
operands are R / theta (entries in [-1, 1], since theta >= ||R||_2) and g,
rounded to fp16; the product is scaled back by theta. R, the Ritz step, the
Lanczos scale and every sum stay wide.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .filters import ns_filter
from .linalg import cholqr
from .precision import round_f16
from .rng import lanczos_start

CUBIC = (1.5, -0.5)


@dataclass
class PSDInfo:
    n_deflated: int
    n_positive: int
    theta: float
    ritz: np.ndarray


def lanczos_scale(apply_b, n: int, seed: int = 0, steps: int = 20) -> float:
    """Upper estimate of sqrt(lambda_max(B)) for a PSD operator B (App. E.1)."""
    m = min(steps, n)
    q = lanczos_start(seed, n)
    basis = [q / np.linalg.norm(q)]
    alpha, beta = [], []
    for j in range(m):
        w = apply_b(basis[j])
        a_j = float(basis[j] @ w)
        w = w - a_j * basis[j]
        if j > 0:
            w = w - beta[j - 1] * basis[j - 1]
        qm = np.stack(basis, axis=1)
        for _ in range(2):
            w = w - qm @ (qm.T @ w)
        alpha.append(a_j)
        if j == m - 1:
            break
        b_j = float(np.linalg.norm(w))
        if b_j == 0.0:
            break
        beta.append(b_j)
        basis.append(w / b_j)
    kk = len(alpha)
    t = np.diag(alpha) + np.diag(beta[:kk - 1], 1) + np.diag(beta[:kk - 1], -1)
    evals, evecs = np.linalg.eigh(t)
    rho = float(evals[-1])
    v = np.stack(basis[:kk], axis=1) @ evecs[:, -1]
    res = float(np.linalg.norm(apply_b(v) - rho * v))
    return float(np.sqrt(max(rho + res, 0.0)))


def ritz_order(lam: np.ndarray) -> np.ndarray:
    idx = np.arange(lam.size)
    return np.lexsort((idx, -lam, -np.abs(lam)))


def residual_scale(r: np.ndarray, scale: str, seed: int, lanczos_steps: int) -> float:
    """theta: the Lanczos upper estimate of ||R||_2 (App. E.1) or ||R||_F."""
    if scale == "lanczos":
        return lanczos_scale(lambda x: r @ (r @ x), r.shape[0], seed, lanczos_steps)
    if scale == "frobenius":
        return float(np.linalg.norm(r))
    raise ValueError(f"unknown scale {scale!r}")


def psd_project_deflated(z, basis, *, table=None, steps=10, gamma=1.1, tau=0.0,
                         window=0, subspace_iters=1, seed=0, lanczos_steps=20, mode="exact",
                         scale="lanczos"):
    """Alg. 2. z: symmetric (n x n); basis: orthonormal (n x K).
    mode: the sign filter's arithmetic, "exact" or "f16" (filters.ns_filter).
    scale: "lanczos" (App. E.1) or "frobenius". Returns (P, V_next, info)."""
    z = np.asarray(z, dtype=np.float64)
    v = np.asarray(basis, dtype=np.float64)
    n, kk = v.shape
    table = [CUBIC] * steps if table is None else table
    for _ in range(subspace_iters - 1):
        v = cholqr(z @ v)
    zt = z @ v
    t = v.T @ zt
    t = 0.5 * (t + t.T)
    lam, e = np.linalg.eigh(t)
    u = v @ e
    order = ritz_order(lam)
    lam, u = lam[order], u[:, order]
    s = np.abs(lam)
    if tau > 0.0:
        r = max(1, min(window, kk))
        n_def = int(np.count_nonzero(s > tau * s[0])) if s[r - 1] < tau * s[0] else 0
    else:
        n_def = kk
    if n_def > 0:
        ui, li = u[:, :n_def], lam[:n_def]
        res = z - (ui * li) @ ui.T
        theta = residual_scale(res, scale, seed, lanczos_steps)
        x0 = (res / theta if theta > 0 else np.zeros_like(res)) \
            + (ui * np.sign(li)) @ ui.T / gamma
        g = ns_filter(x0, table, mode)
        p = 0.5 * (res + restore_product(res, g, theta, mode)) + (ui * np.maximum(li, 0.0)) @ ui.T
        n_pos = int(np.count_nonzero(li > 0))
    else:
        theta = residual_scale(z, scale, seed, lanczos_steps)
        x0 = z / theta if theta > 0 else np.zeros_like(z)
        g = ns_filter(x0, table, mode)
        p = 0.5 * (z + restore_product(z, g, theta, mode))
        n_pos = 0
    p = 0.5 * (p + p.T)
    return p, cholqr(zt), PSDInfo(n_def, n_pos, theta, lam)


def psd_project(z, *, table=None, steps=10, seed=0, lanczos_steps=20, mode="exact", scale="lanczos"):
    """Undeflated baseline projection (eq:baseline_projection), symmetrized."""
    z = np.asarray(z, dtype=np.float64)
    table = [CUBIC] * steps if table is None else table
    theta = residual_scale(z, scale, seed, lanczos_steps)
    x0 = z / theta if theta > 0 else np.zeros_like(z)
    g = ns_filter(x0, table, mode)
    p = 0.5 * (z + restore_product(z, g, theta, mode))
    return 0.5 * (p + p.T), theta


def restore_product(r: np.ndarray, g: np.ndarray, theta: float, mode: str) -> np.ndarray:
    """R g, the product that restores the sign filter's output (Alg. 2,
    eq:baseline_projection); in fp16 mode theta fp16(R / theta) fp16(g)."""
    if mode != "f16":
        return r @ g
    if theta <= 0.0:
        return np.zeros_like(r)
    return theta * (round_f16(r / theta) @ round_f16(g))


def psd_exact(z: np.ndarray) -> np.ndarray:
    """Pi_+(Z) = V max(Lambda, 0) V^T from a full eigendecomposition (eq:psd_sign)."""
    lam, v = np.linalg.eigh(np.asarray(z, dtype=np.float64))
    return (v * np.maximum(lam, 0.0)) @ v.T
