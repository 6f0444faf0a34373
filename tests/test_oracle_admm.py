"""Pins of oracle.admm (eq:admm_iter, eq:admm_eta) against closed forms and the
paper's claim for ADMM with the deflated projection (Sec. 3.3)."""
import numpy as np

import workloads
from oracle import admm, psd


def test_maxcut_sdp_known_optima():
    # Complete graph K_6: the optimum is the regular-simplex Gram, value n^2 / 4.
    # Cycle C_5: value (5 / 2)(1 + cos(pi / 5)). Exact projections; the primal
    # and dual objectives meet and the KKT residual vanishes.
    for w, want in [(np.ones((6, 6)) - np.eye(6), 9.0),
                    (np.roll(np.eye(5), 1, 1) + np.roll(np.eye(5), -1, 1), 2.5 * (1 + np.cos(np.pi / 5)))]:
        c = admm.maxcut_cost(w)
        b = np.ones(w.shape[0])
        x, s, y, etas = admm.admm_diag(c, b, 3000, admm.exact_projector)
        assert abs(-np.sum(c * x) - want) < 1e-9
        assert abs(-(b @ y) - want) < 1e-9
        assert etas[-1] < 1e-12
        np.testing.assert_allclose(np.diag(x), 1.0, atol=1e-12)


def test_kkt_eta_terms():
    # eta is the max of the three scaled residuals, each checked on its own
    c = np.diag([1.0, 2.0])
    b = np.array([1.0, 1.0])
    x = np.diag([2.0, 1.0])                      # primal residual (1, 0)
    y = np.array([0.0, 0.0])
    s = c.copy()                                 # dual residual 0
    want_primal = 1.0 / (1 + np.sqrt(2))
    pobj, dobj = 4.0, 0.0
    want_gap = abs(pobj - dobj) / (1 + pobj + dobj)
    assert abs(admm.kkt_eta(c, b, x, y, s) - max(want_primal, want_gap)) < 1e-15


def test_projector_schedule():
    case = workloads.planted_maxcut(120, case_id=1)
    z = case.c.astype(np.float64) - np.eye(120)
    base = admm.DeflatedProjector(None)
    np.testing.assert_array_equal(base(z), psd.psd_project(z, steps=10)[0])
    proj = admm.DeflatedProjector(case.basis0.astype(np.float64), tau=0.1, window=case.window, warmup=3)
    for _ in range(3):
        proj(z)
    assert proj.n_deflated == [0, 0, 0]            # gate held closed during the warm-up
    v = proj.basis.copy()
    p = proj(z)                                    # then Alg. 2 with the tracked basis
    want, vnext, info = psd.psd_project_deflated(z, v, steps=10, gamma=1.1, tau=0.1, window=case.window)
    np.testing.assert_array_equal(p, want)
    np.testing.assert_allclose(proj.basis, vnext, rtol=0, atol=1e-12)   # BLAS rounding may differ
    assert proj.n_deflated[-1] == info.n_deflated


def test_deflation_lowers_kkt_residual():
    # The paper's SDP result (Sec. 3.3): with the same fixed filter budget the
    # deflated projection lets ADMM keep converging where the undeflated one
    # stalls. Planted-cut instance, 250 iterations, sigma = 1, gate off for 100.
    case = workloads.planted_maxcut(120, case_id=2)
    c, b = case.c.astype(np.float64), case.b.astype(np.float64)
    _, _, _, e_base = admm.admm_diag(c, b, 250, admm.DeflatedProjector(None))
    proj = admm.DeflatedProjector(case.basis0.astype(np.float64), tau=0.1, window=case.window, warmup=100)
    _, _, _, e_def = admm.admm_diag(c, b, 250, proj)
    _, _, _, e_exact = admm.admm_diag(c, b, 250, admm.exact_projector)
    assert max(proj.n_deflated[100:]) > 0
    assert e_def[-1] < 0.5 * e_base[-1]
    assert e_exact[-1] < e_def[-1]
