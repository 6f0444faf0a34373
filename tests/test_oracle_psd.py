"""Pins of oracle.psd (Alg. 2, App. E.1) against closed forms and bounds."""
import numpy as np
import pytest

import workloads
from oracle import psd
from oracle.filters import bjorck_bowie, scalar_compose


def sym_case(seed, n, lam):
    g = np.random.default_rng(seed)
    q, _ = np.linalg.qr(g.standard_normal((n, n)))
    return (q * lam) @ q.T, q


@pytest.mark.parametrize("seed", range(6))
def test_lanczos_is_an_upper_estimate(seed):
    # App. E.1: theta >= ||Z||_2 (heuristic; never violated on these inputs) and close to it.
    g = np.random.default_rng(seed)
    n = 150
    lam = np.concatenate([g.uniform(5, 10, 3) * g.choice([-1, 1], 3), g.uniform(-1, 1, n - 3)])
    z, _ = sym_case(seed, n, lam)
    theta = psd.lanczos_scale(lambda x: z @ (z @ x), n, seed)
    norm2 = np.abs(np.linalg.eigvalsh(z)).max()
    assert norm2 <= theta <= norm2 * 1.05


def test_lanczos_small_n_is_exact_and_zero_is_zero():
    g = np.random.default_rng(3)
    a = g.standard_normal((8, 8))
    z = a + a.T
    theta = psd.lanczos_scale(lambda x: z @ (z @ x), 8)
    assert abs(theta - np.abs(np.linalg.eigvalsh(z)).max()) < 1e-6
    zero = np.zeros((10, 10))
    assert psd.lanczos_scale(lambda x: zero @ x, 10) == 0.0


def test_ritz_order_rule():
    lam = np.array([1.0, -3.0, 3.0, 0.5, -0.5, 2.0])
    assert list(psd.ritz_order(lam)) == [2, 1, 5, 0, 3, 4]


def test_baseline_scalarized_closed_form():
    # eq:psd_error_base: in the eigenbasis of Z the output is 1/2 lam (1 + p^L(lam / theta)).
    n = 40
    g = np.random.default_rng(2)
    lam = np.concatenate([[30.0, -20.0], g.uniform(-1, 1, n - 2)])
    z, q = sym_case(0, n, lam)
    table = [bjorck_bowie(1)] * 8
    p, theta = psd.psd_project(z, table=table)
    want = (q * (0.5 * lam * (1 + scalar_compose(lam / theta, table)))) @ q.T
    np.testing.assert_allclose(p, want, atol=1e-11)


def test_baseline_converges_to_projection():
    n = 30
    g = np.random.default_rng(5)
    lam = g.uniform(0.05, 1, n) * g.choice([-1, 1], n)
    z, _ = sym_case(1, n, lam)
    p, _ = psd.psd_project(z, table=[bjorck_bowie(1)] * 40)
    np.testing.assert_allclose(p, psd.psd_exact(z), atol=1e-10)


@pytest.mark.parametrize("gamma", [1.0, 1.01, 1.1, 2.0])
def test_exact_deflation_is_gamma_independent_and_scalarized(gamma):
    # Prop. 2: with exact eigenpairs the output does not depend on gamma, the head is
    # restored exactly and the tail passes the filter with the residual scale.
    n, k = 40, 4
    g = np.random.default_rng(8)
    lam = np.concatenate([[50.0, -40.0, 30.0, -25.0], g.uniform(-1, 1, n - k)])
    z, q = sym_case(3, n, lam)
    table = [bjorck_bowie(1)] * 6
    p, vnext, info = psd.psd_project_deflated(z, q[:, :k], table=table, gamma=gamma)
    assert info.n_deflated == 4 and info.n_positive == 2
    tail = lam[k:]
    f = np.concatenate([np.maximum(lam[:k], 0),
                        0.5 * tail * (1 + scalar_compose(tail / info.theta, table))])
    np.testing.assert_allclose(p, (q * f) @ q.T, atol=1e-10)
    # theta estimates ||R||_2 = max |tail|
    assert np.abs(tail).max() <= info.theta <= np.abs(tail).max() * 1.05
    # next basis spans Z V = span(q_k)
    np.testing.assert_allclose(vnext @ vnext.T, q[:, :k] @ q[:, :k].T, atol=1e-10)


def test_prop2_ratio_bound():
    # eq:deflated_psd_ratio with exact eigenpairs, theta = exact norms (both sides
    # computed here from the oracle's own theta, which is an upper estimate).
    n, k = 60, 3
    g = np.random.default_rng(12)
    lam = np.concatenate([[80.0, -60.0, 45.0], g.uniform(-1, 1, n - k)])
    lam[-1] = 0.02
    z, q = sym_case(4, n, lam)
    target = psd.psd_exact(z)
    for L in range(1, 7):
        table = [bjorck_bowie(1)] * L
        pb, theta = psd.psd_project(z, table=table)
        pd, _, info = psd.psd_project_deflated(z, q[:, :k], table=table)
        ell = np.abs(lam).min() / theta
        alpha_ell = np.abs(lam).min() / info.theta
        eb = np.linalg.norm(pb - target, 2)
        ed = np.linalg.norm(pd - target, 2)
        bound = ((1 - alpha_ell ** 2) / (1 - ell ** 2)) ** (2 ** L)
        assert ed <= bound * eb * (1 + 1e-9) + 1e-12
        assert ed < eb


def test_gate_and_fallback_to_baseline():
    n, k = 40, 6
    g = np.random.default_rng(6)
    lam = np.concatenate([[50.0, -40.0], g.uniform(-1, 1, n - 2)])
    z, q = sym_case(5, n, lam)
    basis = np.linalg.qr(q[:, :k] + 1e-3 * g.standard_normal((n, k)))[0]
    p, _, info = psd.psd_project_deflated(z, basis, tau=0.1, window=4, steps=8)
    assert info.n_deflated == 2 and info.n_positive == 1
    # a gate that does not fire gives the baseline bitwise
    flat = np.concatenate([g.uniform(0.5, 1, 6) * g.choice([-1, 1], 6), g.uniform(-0.4, 0.4, n - 6)])
    z2, q2 = sym_case(7, n, flat)
    p2, _, info2 = psd.psd_project_deflated(z2, q2[:, :k], tau=0.1, window=4, steps=8)
    pb, _ = psd.psd_project(z2, steps=8)
    assert info2.n_deflated == 0
    np.testing.assert_array_equal(p2, pb)


def test_deflation_lowers_error_on_small_config4_like():
    c = workloads.small_psd(256, k=8, n_dom=4, dom=(200.0, 1000.0))
    z = c.z.astype(np.float64)
    target = psd.psd_exact(z)
    pb, _ = psd.psd_project(z, steps=c.steps)
    pd, _, info = psd.psd_project_deflated(z, c.qwarm, steps=c.steps, gamma=c.gamma,
                                           subspace_iters=c.subspace_iters)
    assert np.linalg.norm(pd - target) < 0.1 * np.linalg.norm(pb - target)
    np.testing.assert_allclose(np.sort(np.abs(info.ritz[:4])),
                               np.sort(np.abs(c.lam[np.argsort(-np.abs(c.lam))[:4]])), rtol=1e-6)


# --- fp16 contract of the sign filter ----------------------------------------------
def test_f16_filter_step_is_exact_on_dyadic_input():
    # A diagonal X with dyadic entries keeps every operand, product and
    # coefficient combination exactly representable: the fp16 contract must
    # then equal exact arithmetic bit for bit (no rounding point is missing
    # an operand, and none is applied to a wide value).
    from oracle.filters import ns_filter
    x = np.diag([0.5, -0.25, 0.75, 0.125, 0.0, -1.0])
    for table in ([(1.5, -0.5)], [(1.875, -1.25, 0.375)]):
        np.testing.assert_array_equal(ns_filter(x, table, "f16"), ns_filter(x, table))


def test_f16_projection_within_the_fp16_error_of_exact():
    # Operand rounding of 2^-11 relative, grown by the filter's slope, moves
    # the output far less than the filter's own error: on a deflated case the
    # fp16-contract projection stays within 1e-2 of the exact-arithmetic one
    # and shares its bookkeeping, and differs from it (the contract is applied).
    case = workloads.small_psd(160, k=8, case_id=12)
    z = case.z.astype(np.float64)
    q = case.qwarm.astype(np.float64)
    p64, v64, i64 = psd.psd_project_deflated(z, q, steps=case.steps, gamma=case.gamma,
                                             subspace_iters=case.subspace_iters)
    p16, v16, i16 = psd.psd_project_deflated(z, q, steps=case.steps, gamma=case.gamma,
                                             subspace_iters=case.subspace_iters, mode="f16")
    err = np.linalg.norm(p16 - p64) / np.linalg.norm(p64)
    assert 0 < err < 1e-2
    assert (i16.n_deflated, i16.n_positive) == (i64.n_deflated, i64.n_positive)
    np.testing.assert_array_equal(v16, v64)   # the basis update does not involve the filter



def test_f16_restore_product_rounds_normalized_operands():
    # The fp16 restore product rounds R / theta (not R) and g. With R = 3 F,
    # theta = 3 and F, g on the fp16 grid, both operands survive rounding,
    # so the product equals the exact one bit for bit; rounding R itself
    # would not (3 F needs up to 13 significant bits).
    from oracle.precision import round_f16
    rng = np.random.default_rng(7)
    f = round_f16(rng.uniform(-1, 1, (24, 24)))
    g = round_f16(rng.uniform(-1, 1, (24, 24)))
    r = 3.0 * f
    assert not np.array_equal(round_f16(r), r)
    np.testing.assert_array_equal(psd.restore_product(r, g, 3.0, "f16"), r @ g)
    # a zero scale gives a zero product; exact mode is the plain product
    np.testing.assert_array_equal(psd.restore_product(r, g, 0.0, "f16"), np.zeros_like(r))
    np.testing.assert_array_equal(psd.restore_product(r, g, 3.0, "exact"), r @ g)


def test_f16_restore_product_within_the_operand_rounding_bound():
    # |fl16(a) - a| <= 2^-11 |a| per operand, so
    # ||theta (R~ g~) - R g||_F <= 2^-11 theta (||R/theta||_F ||g~||_2 + ||R/theta||_2 ||g||_F);
    # the error is nonzero on generic operands (the rounding is applied).
    rng = np.random.default_rng(8)
    a = rng.standard_normal((64, 64))
    r = a + a.T
    theta = 1.01 * np.linalg.norm(r, 2)
    g = np.tanh(rng.standard_normal((64, 64)))
    err = np.linalg.norm(psd.restore_product(r, g, theta, "f16") - r @ g)
    from oracle.precision import round_f16
    bound = 2.0 ** -11 * theta * (np.linalg.norm(r / theta) * np.linalg.norm(round_f16(g), 2)
                                  + np.linalg.norm(r / theta, 2) * np.linalg.norm(g))
    assert 0 < err <= bound


# --- Frobenius scale ----------------------------------------------------------------
def test_frobenius_scale_closed_form_and_convergence():
    # With exact Ritz pairs (the basis spans the dominant eigenvectors), the
    # residual is the rest of the spectrum: theta = sqrt(sum_{i not in I}
    # lam_i^2) >= ||R||_2, so X0's spectrum lies in [-1, 1] and the classical
    # filter converges to Pi_+ with enough steps.
    n, k = 48, 4
    g = np.random.default_rng(31)
    lam = np.concatenate([[60.0, -45.0, 30.0, 20.0], g.uniform(-1, 1, n - k)])
    z, q = sym_case(31, n, lam)
    order = np.argsort(-np.abs(lam))
    basis = q[:, order[:k]]
    p, _, info = psd.psd_project_deflated(z, basis, steps=60, scale="frobenius")
    tail = np.delete(lam, order[:k])
    np.testing.assert_allclose(info.theta, np.sqrt(np.sum(tail ** 2)), rtol=1e-12)
    assert info.theta >= np.max(np.abs(tail))
    np.testing.assert_allclose(p, psd.psd_exact(z), atol=1e-6 * np.linalg.norm(z))
    # the undeflated form scales by ||Z||_F
    pb, theta_b = psd.psd_project(z, steps=5, scale="frobenius")
    np.testing.assert_allclose(theta_b, np.linalg.norm(z), rtol=1e-12)
    with pytest.raises(ValueError):
        psd.psd_project(z, steps=1, scale="spectral")
