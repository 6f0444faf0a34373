"""Pins of oracle.muon (Alg. 1, Alg. 3) against invariants, bounds and brute force."""
import numpy as np
import pytest

import workloads
from oracle import filters, muon, rng
from oracle.filters import bjorck_bowie, ns_filter, scalar_compose


def haar(g, n, k):
    q, r = np.linalg.qr(g.standard_normal((n, k)))
    return q * np.sign(np.diag(r))


def spiked(g, n, m, head, tail_lo=1e-3):
    sig = np.concatenate([head, np.sort(10 ** g.uniform(np.log10(tail_lo), 0, m - len(head)))[::-1]])
    u, v = haar(g, n, m), haar(g, m, m)
    return (u * sig) @ v.T, u, sig, v


# --- Alg. 3 -----------------------------------------------------------------------
def test_rsvd_exact_when_rank_fits_sketch():
    # A matrix of rank <= r' is captured exactly by the sketch (App. D bounds with sigma_{k+1} = 0).
    g = np.random.default_rng(0)
    n, m, rank = 60, 30, 6
    a = haar(g, n, rank) @ np.diag([9, 7, 5, 3, 2, 1.0]) @ haar(g, m, rank).T
    omega = rng.sketch(0, 0, m, 10)
    u, s, v = muon.randomized_svd(a, 4, 10, 0, omega)
    uu, ss, vvt = np.linalg.svd(a)
    np.testing.assert_allclose(s, ss[:4], rtol=1e-10)
    np.testing.assert_allclose((u * s) @ v.T, (uu[:, :4] * ss[:4]) @ vvt[:4], atol=1e-10)


@pytest.mark.parametrize("power_iters", [0, 1, 2])
def test_rsvd_singular_values_within_gu_bound(power_iters):
    # App. D: sigma_i >= s_i >= sigma_i / sqrt(1 + (sigma_{k+1}/sigma_i)^(2(2J+1)) ||O2 O1^+||^2)
    g = np.random.default_rng(10 + power_iters)
    n, m, k, p = 120, 80, 5, 5
    a, u, sig, v = spiked(g, n, m, [30, 20, 12, 8, 5], tail_lo=1e-2)
    sig = sig.copy()
    for seed in range(10):
        omega = rng.sketch(seed, 0, m, k + p)
        _, s, _ = muon.randomized_svd(a, k, k + p, power_iters, omega)
        o1 = v[:, :k].T @ omega
        o2 = v[:, k:].T @ omega
        w = np.linalg.norm(o2 @ np.linalg.pinv(o1), 2)
        for i in range(k):
            lower = sig[i] / np.sqrt(1 + (sig[k] / sig[i]) ** (2 * (2 * power_iters + 1)) * w ** 2)
            assert sig[i] * (1 + 1e-9) >= s[i] >= lower * (1 - 1e-9)


def test_rsvd_head_subspace_angle_bound():
    # App. D: sin(theta_i) <= (sigma_{k+1}/sigma_i)^(2J+1) ||O2 O1^+||, left head subspace.
    g = np.random.default_rng(4)
    n, m, k, p, J = 100, 70, 4, 6, 1
    a, u, sig, v = spiked(g, n, m, [40, 25, 15, 9], tail_lo=1e-2)
    omega = rng.sketch(3, 0, m, k + p)
    uh, _, _ = muon.randomized_svd(a, k, k + p, J, omega)
    o1, o2 = v[:, :k].T @ omega, v[:, k:].T @ omega
    w = np.linalg.norm(o2 @ np.linalg.pinv(o1), 2)
    # largest canonical angle between span(uh) and span(u_k)
    sin_max = np.linalg.norm(uh - u[:, :k] @ (u[:, :k].T @ uh), 2)
    assert sin_max <= (sig[k] / sig[k - 1]) ** (2 * J + 1) * w * (1 + 1e-9)


# --- Alg. 1 -----------------------------------------------------------------------
def test_gate_rank_rule():
    s = np.array([10.0, 5.0, 2.0, 1.0, 0.5])
    assert muon.deflation_rank(s, 5, 0.1) == 3           # fires (0.5 < 1); s_i > 1 strictly
    assert muon.deflation_rank(s, 3, 0.1) == 0           # s_3 = 2 >= 1: no fire
    assert muon.deflation_rank(s, 4, 0.0) == 4           # fixed rank
    assert muon.deflation_rank(s, 0, 0.1) == 0
    assert muon.deflation_rank(np.array([10, 1.0, 0.99]), 3, 0.1) == 1   # equality excluded
    assert muon.deflation_rank(np.zeros(4), 4, 0.1) == 0


@pytest.mark.parametrize("gamma", [1.0, 1.01, 1.1, 2.0])
def test_exact_deflation_preserves_target(gamma):
    # eq:identities: polar(R/||R|| + gamma^-1 U_k V_k^T) = polar(M) for exact triplets.
    g = np.random.default_rng(1)
    a, u, sig, v = spiked(g, 40, 20, [30, 10, 4])
    x0, _ = muon.deflated_init(a, u, sig, v, 3, gamma)
    np.testing.assert_allclose(muon.polar_exact(x0), muon.polar_exact(a), atol=1e-12)


def test_zero_matrix_maps_to_zero():
    x = np.zeros((2, 12, 20))
    for k in (0, 3):
        out, info = muon.msign_deflated(x, k, [filters.MUON_QUINTIC] * 5)
        assert np.all(out == 0)


def test_gate_off_is_baseline_bitwise():
    # Sec. 2.2: when the gate does not fire the method reduces exactly to Muon.
    c = workloads.small_muon(2, 24, 40, k=3, spikes=[2.0, 1.9, 1.8])
    table = c.coeffs
    base = muon.msign(c.x64, table)
    out, info = muon.msign_deflated(c.x64, 3, table, tau=0.1)
    assert info.k_eff == [0, 0]
    np.testing.assert_array_equal(out, base)


def test_transpose_identity_exact():
    # App. D, "Grouping": polar(M^T) = polar(M)^T; the method transposes wide inputs.
    c = workloads.small_muon(2, 20, 33, k=3)
    table = c.coeffs
    out, info = muon.msign_deflated(c.x64, 3, table)
    out_t, info_t = muon.msign_deflated(np.transpose(c.x64, (0, 2, 1)).copy(), 3, table)
    assert info.transposed and not info_t.transposed
    np.testing.assert_allclose(out, np.transpose(out_t, (0, 2, 1)), atol=1e-12)


def test_pipeline_with_exact_head_matches_scalarized_closed_form():
    # rank(M) = k + (tail) and r' covers the head: with J >= 1 the estimated head is
    # exact to rounding, and the output equals U diag(p^L(x_i)) V^T with
    # x = (1/gamma for the head, sigma_i / ||R||_F for the tail).
    g = np.random.default_rng(9)
    n, m, k = 50, 12, 3
    sig = np.array([40.0, 20.0, 10.0, 1.0, 0.8, 0.5, 0.3, 0.2, 0.1, 0.05, 0.02, 0.01])
    u, v = haar(g, n, m), haar(g, m, m)
    a = (u * sig) @ v.T
    table = [bjorck_bowie(2)] * 5
    out, info = muon.msign_deflated(a[None], k, table, oversample=9, power_iters=2, gamma=1.01)
    nu = np.linalg.norm(sig[k:])
    x = np.concatenate([np.full(k, 1 / 1.01), sig[k:] / nu])
    want = (u * scalar_compose(x, table)) @ v.T
    np.testing.assert_allclose(out[0], want, atol=1e-9)
    np.testing.assert_allclose(info.nu[0], nu, rtol=1e-12)


def test_tail_far_below_the_spike_is_kept():
    # Alg. 1 as written has no floor on nu: a full-rank input whose tail sits
    # 1e-6 below the spike (64 x 200, spike 1e6 over a tail in [1e-2, 1],
    # k = 1) keeps its tail. The deflated output is full rank and close to
    # polar(M); the undeflated filter cannot resolve the tail at all.
    g = np.random.default_rng(5)
    m, n = 64, 200
    sig = np.concatenate([[1e6], np.sort(10 ** g.uniform(-2, 0, m - 1))[::-1]])
    a = (haar(g, m, m) * sig) @ haar(g, n, m).T
    table = [filters.MUON_QUINTIC] * 5
    target = muon.polar_exact(a[None])[0]
    out, info = muon.msign_deflated(a[None], 1, table, power_iters=2)
    sv = np.linalg.svd(out[0], compute_uv=False)
    assert sv.min() > 0.3 and np.linalg.matrix_rank(out[0]) == m
    err = np.linalg.norm(out[0] - target) / np.linalg.norm(target)
    base = muon.msign(a[None], table)[0]
    err_base = np.linalg.norm(base - target) / np.linalg.norm(target)
    assert err < 0.2 < 0.9 < err_base
    np.testing.assert_allclose(info.nu[0], np.linalg.norm(sig[1:]), rtol=1e-6)


def test_gate_window_separate_from_k():
    # Alg. 1's gate over a window of r estimated values, capped at k.
    s = np.array([10.0, 5.0, 2.0, 1.5, 0.5, 0.2])
    assert muon.deflation_rank(s, 6, 0.1, r=6) == 4       # s_6 < 1: the four values above 1
    assert muon.deflation_rank(s, 2, 0.1, r=6) == 2       # capped at k
    assert muon.deflation_rank(s, 6, 0.1, r=4) == 0       # s_4 = 1.5 >= 1: no fire
    assert muon.deflation_rank(s, 3, 0.1) == 0            # window defaults to k
    # through the pipeline: a window of 6 sketched values deflates the 3 spikes
    case = workloads.small_muon(1, 60, 150, k=6, spikes=[50, 30, 20, 1.0, 0.9, 0.8], bulk=(1e-3, 0.5),
                                case_id=44)
    _, info = muon.msign_deflated(case.x64, 2, case.coeffs, tau=0.1, window=6)
    assert info.k_eff == [2] and info.rprime == 14
    _, info = muon.msign_deflated(case.x64, 6, case.coeffs, tau=0.1, window=6)
    assert info.k_eff == [3]


def test_explicit_restore_matches_scalarized_closed_form():
    # Explicit restore (eq:identities): the head is added after the filter, so
    # its singular values are exactly 1 and the tail's are p^L(sigma_i / ||R||_F).
    g = np.random.default_rng(19)
    n, m, k = 50, 12, 3
    sig = np.array([40.0, 20.0, 10.0, 1.0, 0.8, 0.5, 0.3, 0.2, 0.1, 0.05, 0.02, 0.01])
    u, v = haar(g, n, m), haar(g, m, m)
    a = (u * sig) @ v.T
    table = [bjorck_bowie(2)] * 5
    out, info = muon.msign_deflated(a[None], k, table, oversample=9, power_iters=2, restore="explicit")
    nu = np.linalg.norm(sig[k:])
    x = np.concatenate([np.ones(k), scalar_compose(sig[k:] / nu, table)])
    want = (u * x) @ v.T
    np.testing.assert_allclose(out[0], want, atol=1e-9)
    # the padded form with a huge gamma leaves the head out of the filter: it
    # differs from the explicit form by exactly U_k V_k^T
    pad, _ = muon.msign_deflated(a[None], k, table, oversample=9, power_iters=2, gamma=1e30)
    np.testing.assert_allclose(out[0] - pad[0], u[:, :k] @ v[:, :k].T, atol=1e-9)


def test_explicit_restore_converges_to_polar_and_k0_is_baseline():
    g = np.random.default_rng(23)
    a, *_ = spiked(g, 40, 16, [30.0, 10.0], tail_lo=0.05)
    # 20 classical steps resolve the tail (sigma_min / ||R||_F = 0.056). Many more
    # would not stay converged: the head directions of R / nu are rounding-level
    # (1e-16), the filter grows them by about 1.5 per step, and after ~60 steps
    # they rejoin the restored head. The padded form has no such drift.
    table = [bjorck_bowie(1)] * 20
    # r' = m: the estimated head is exact, so the split is the exact one of eq:identities
    out, _ = muon.msign_deflated(a[None], 2, table, oversample=14, restore="explicit")
    np.testing.assert_allclose(out[0], muon.polar_exact(a[None])[0], atol=1e-8)
    base = muon.msign(a[None], table[:5])
    expl, _ = muon.msign_deflated(a[None], 0, table[:5], restore="explicit")
    assert np.array_equal(base, expl)


def test_deflation_lowers_error_on_config1():
    # Sec. 3 claim (empirical with Muon's coefficients): deflation lowers the error to polar(M).
    c = workloads.config1()
    target = muon.polar_exact(c.x64)
    base = muon.msign(c.x64, c.coeffs)
    out, info = muon.msign_deflated(c.x64, c.k, c.coeffs, oversample=c.oversample,
                                    power_iters=c.power_iters, gamma=c.gamma)
    eb = np.linalg.norm(base - target) / np.linalg.norm(target)
    ed = np.linalg.norm(out - target) / np.linalg.norm(target)
    assert ed < 0.7 * eb
    # the estimated head is accurate (App. D, head accuracy)
    np.testing.assert_allclose(info.s[0], c.spectra[0][:c.k], rtol=1e-4)


def test_bf16_mode_outputs_are_bf16_and_close():
    from oracle.precision import round_bf16
    c = workloads.small_muon(2, 32, 96, dtype="bf16", k=4, bulk=(1e-2, 1.0))
    e, _ = muon.msign_deflated(c.x64, 4, c.coeffs)
    b, _ = muon.msign_deflated(c.x64, 4, c.coeffs, mode="bf16")
    np.testing.assert_array_equal(round_bf16(b), b)
    rel = np.linalg.norm(b - e) / np.linalg.norm(e)
    assert 1e-6 < rel < 3e-2
