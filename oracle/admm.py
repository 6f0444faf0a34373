"""Three-block ADMM for the standard-form SDP pair (App. E.1), on the CPU.

Primal  min <C, X>  s.t.  A X = b,  X PSD;   dual  max b^T y  s.t.  A* y + S = C,  S PSD
(eq:sdp_pair). One iteration with penalty sigma (eq:admm_iter):
    y = (A A*)^-1 (b / sigma - A(X / sigma + S - C))
    Z = C - A* y - X / sigma,   S = Pi_+(Z)
    X = X + sigma (S + A* y - C)
This module takes diagonal constraints, the max-cut relaxation's: A X = diag(X),
A* y = Diag(y), so A A* = I and the y-update is elementwise. The projection is
a callable (the exact Pi_+ from eigh, or the deflated projection of Alg. 2
with a tracked basis, see DeflatedProjector). KKT residual: the first three,
eigenvalue-free terms of eq:admm_eta.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from .psd import psd_exact, psd_project, psd_project_deflated


def maxcut_cost(w: np.ndarray) -> np.ndarray:
    """C = -L / 4 for the max-cut relaxation max (1/4) <L, X> of a weighted
    graph with symmetric weights w (zero diagonal), L = Diag(w 1) - w."""
    w = np.asarray(w, dtype=np.float64)
    lap = np.diag(w.sum(axis=1)) - w
    return -0.25 * lap


def kkt_eta(c, b, x, y, s) -> float:
    """max of the primal, dual and gap terms of eq:admm_eta for A X = diag(X)."""
    nb, nc = float(np.linalg.norm(b)), float(np.linalg.norm(c))
    primal = float(np.linalg.norm(np.diag(x) - b)) / (1.0 + nb)
    dual = float(np.linalg.norm(np.diag(y) + s - c)) / (1.0 + nc)
    pobj, dobj = float(np.sum(c * x)), float(b @ y)
    gap = abs(pobj - dobj) / (1.0 + abs(pobj) + abs(dobj))
    return max(primal, dual, gap)


@dataclass
class DeflatedProjector:
    """Alg. 2 inside ADMM: one block step and Rayleigh-Ritz per projection on
    a tracked basis of K columns, the gate (tau, window r) held closed for the
    first `warmup` projections while the basis settles (Sec. 3.3), the basis
    replaced by CholQR(Z V) after every projection. k = 0 gives the undeflated
    baseline (eq:baseline_projection)."""
    basis: np.ndarray | None
    tau: float = 0.1
    window: int = 1
    gamma: float = 1.1
    steps: int = 10
    warmup: int = 100
    mode: str = "exact"
    calls: int = 0
    n_deflated: list = field(default_factory=list)
    ritz: list = field(default_factory=list)

    def __call__(self, z: np.ndarray) -> np.ndarray:
        if self.basis is None:
            p, _ = psd_project(z, steps=self.steps, mode=self.mode)
            self.n_deflated.append(0)
        else:
            tau = self.tau if self.calls >= self.warmup else 1e-30   # gate closed
            p, self.basis, info = psd_project_deflated(z, self.basis, steps=self.steps, gamma=self.gamma, tau=tau,
                                                       window=self.window, mode=self.mode)
            self.n_deflated.append(info.n_deflated)
            self.ritz.append(info.ritz)
        self.calls += 1
        return p


def admm_diag(c, b, iters, project, *, sigma=1.0, x=None, s=None, y=None):
    """`iters` iterations of eq:admm_iter for A X = diag(X) from (X, S, y)
    (zeros by default). Returns X, S, y and the residual after each iteration."""
    c = np.asarray(c, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    n = c.shape[0]
    x = np.zeros((n, n)) if x is None else np.asarray(x, dtype=np.float64).copy()
    s = np.zeros((n, n)) if s is None else np.asarray(s, dtype=np.float64).copy()
    y = np.zeros(n) if y is None else np.asarray(y, dtype=np.float64).copy()
    etas = []
    for _ in range(iters):
        y = b / sigma - np.diag(x / sigma + s - c)
        z = c - np.diag(y) - x / sigma
        s = project(z)
        x = x + sigma * (s + np.diag(y) - c)
        etas.append(kkt_eta(c, b, x, y, s))
    return x, s, y, etas


def exact_projector(z: np.ndarray) -> np.ndarray:
    return psd_exact(z)
