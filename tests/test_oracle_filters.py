"""Pins of oracle.filters against what the paper and the mathematics fix."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import filters, muon
from oracle.filters import bjorck_bowie, ns_filter, ns_step, scalar_compose, scalar_poly

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def haar(rng, n, k):
    q, r = np.linalg.qr(rng.standard_normal((n, k)))
    return q * np.sign(np.diag(r))


# --- coefficients ------------------------------------------------------------
def test_bjorck_bowie_quintic_is_the_printed_map():
    # eq:muon_ns prints a = 15/8, b = -5/4, c = 3/8; the App. B formula must give them.
    assert bjorck_bowie(2) == [Fraction(15, 8), Fraction(-5, 4), Fraction(3, 8)]


@pytest.mark.parametrize("d", [1, 2, 3, 4, 5])
def test_bjorck_bowie_derivative_identity(d):
    # Lemma 1 (App. B): p_d'(x) = (2d+1) c_d (1 - x^2)^d with c_d = 4^-d C(2d, d).
    from math import comb
    a = bjorck_bowie(d)
    deriv = [a[i] * (2 * i + 1) for i in range(d + 1)]          # coefficients of x^(2i)
    cd = Fraction(comb(2 * d, d), 4 ** d)
    rhs = [(2 * d + 1) * cd * comb(d, i) * (-1) ** i for i in range(d + 1)]
    assert deriv == rhs
    assert sum(a) == 1                                            # p(1) = 1


@pytest.mark.parametrize("d", [1, 2, 3])
def test_residual_identity_and_representation(d):
    # Lemma 1: p_d(x) = x h_d(1 - x^2), h_d(z) = sum_j c_j z^j, and
    # 1 - p_d^2 = (1 - x^2)^(d+1) omega_d(1 - x^2) with 0 < omega_d <= 1.
    from math import comb
    x = np.linspace(0.0, 1.0, 2001)
    z = 1.0 - x * x
    h = sum(comb(2 * j, j) / 4 ** j * z ** j for j in range(d + 1))
    p = scalar_poly(x, bjorck_bowie(d))
    np.testing.assert_allclose(p, x * h, atol=1e-15)
    inner = z[:-1]                                                # exclude x = 1
    omega = (1 - p[:-1] ** 2) / inner ** (d + 1)
    assert np.all(omega > 0) and np.all(omega <= 1 + 1e-12)
    assert np.all(np.diff(p) >= -1e-15) and p.min() >= 0 and p.max() <= 1 + 1e-15


# --- the worked example --------------------------------------------------------
def test_example1_toy_spectrum():
    with open(os.path.join(GOLDEN, "example1.json")) as f:
        gold = json.load(f)
    sig = np.array(gold["singular_values"])
    rng = np.random.default_rng(7)
    u, v = haar(rng, 7, 5), haar(rng, 5, 5)
    m = (u * sig) @ v.T
    table = [bjorck_bowie(2)] * gold["steps"]
    x_base, nrm = muon.deflated_init(m, None, None, None, 0, 1.0)
    x_def, nu = muon.deflated_init(m, u, sig, v, gold["deflated_rank"], gold["gamma"])
    got = {
        "frobenius_norm": nrm,
        "baseline_floor_start": np.linalg.svd(x_base, compute_uv=False).min(),
        "baseline_floor_final": np.linalg.svd(ns_filter(x_base, table), compute_uv=False).min(),
        "residual_norm": nu,
        "alpha": nrm / nu,
        "deflated_floor_start": np.linalg.svd(x_def, compute_uv=False).min(),
        "deflated_floor_final": np.linalg.svd(ns_filter(x_def, table), compute_uv=False).min(),
    }
    for key, spec in gold["printed"].items():
        assert abs(got[key] - spec["value"]) <= spec["abs_tol"], (key, got[key], spec)


# --- scalarization: the matrix step acts on singular values only ---------------
TABLES = {
    "classical": [bjorck_bowie(2)] * 5,
    "muon": [filters.MUON_QUINTIC] * 5,
    "cubic": [bjorck_bowie(1)] * 7,
    "septic": [bjorck_bowie(3)] * 3,
    "varying": [(3.0, -3.2, 1.2), (2.4, -2.0, 0.6), (1.875, -1.25, 0.375)],
}


@pytest.mark.parametrize("name", list(TABLES))
@pytest.mark.parametrize("shape", [(12, 12), (20, 9), (9, 20)])
def test_scalarization(name, shape):
    # App. B (eq:matrix_error_scalarized) and App. D: N^L(U diag(x) V^T) = U diag(p^L(x)) V^T.
    rng = np.random.default_rng(3)
    q = min(shape)
    u, v = haar(rng, shape[0], q), haar(rng, shape[1], q)
    x = np.sort(rng.uniform(1e-3, 1.0, q))
    got = ns_filter((u * x) @ v.T, TABLES[name])
    want = (u * scalar_compose(x, TABLES[name])) @ v.T
    np.testing.assert_allclose(got, want, atol=1e-12)


def test_short_side_gram_equals_literal_map():
    # eq:muon_ns written with the large Gram (X X^T)^i X for a tall X.
    rng = np.random.default_rng(5)
    x = rng.standard_normal((30, 8)) / 8
    a, b, c = filters.MUON_QUINTIC
    big = x @ x.T
    lit = a * x + b * big @ x + c * big @ big @ x
    np.testing.assert_allclose(ns_step(x, (a, b, c)), lit, atol=1e-13)


def test_classical_map_converges_to_polar():
    rng = np.random.default_rng(11)
    m = rng.standard_normal((40, 25))
    x0, _ = muon.deflated_init(m, None, None, None, 0, 1.0)
    got = ns_filter(x0, [bjorck_bowie(2)] * 40)
    np.testing.assert_allclose(got, muon.polar_exact(m), atol=1e-10)


# --- Theorem 1 and the scalarized error -----------------------------------------
@pytest.mark.parametrize("d", [1, 2])
@pytest.mark.parametrize("gamma", [1.0, 1.01, 1.5])
def test_theorem1_bounds(d, gamma):
    rng = np.random.default_rng(100 + d)
    n, mm, k = 24, 16, 3
    sig = np.concatenate([[40.0, 25.0, 12.0], np.sort(10 ** rng.uniform(-2, 0, mm - k))[::-1]])
    u, v = haar(rng, n, mm), haar(rng, mm, mm)
    m = (u * sig) @ v.T
    target = muon.polar_exact(m)
    x_base, nrm = muon.deflated_init(m, None, None, None, 0, gamma)
    x_def, nu = muon.deflated_init(m, u, sig, v, k, gamma)
    ell = sig[-1] / nrm
    alpha = nrm / nu
    phi = min(alpha * ell, 1.0 / gamma)
    # sigma(X_base) in [ell, 1], sigma(X_def) in [phi, 1]
    sb = np.linalg.svd(x_base, compute_uv=False)
    sd = np.linalg.svd(x_def, compute_uv=False)
    assert sb.min() >= ell * (1 - 1e-12) and sb.max() <= 1 + 1e-12
    assert sd.min() >= phi * (1 - 1e-12) and sd.max() <= 1 + 1e-12
    coeffs = bjorck_bowie(d)
    for L in range(7):
        table = [coeffs] * L
        eb = np.linalg.norm(target - ns_filter(x_base, table), 2)
        ed = np.linalg.norm(target - ns_filter(x_def, table), 2)
        # A30: the classical baseline error equals 1 - p^L(ell) exactly
        assert abs(eb - (1 - scalar_compose(ell, table))) < 1e-10
        # eq:deflated_ns_absolute
        assert ed <= (1 - phi ** 2) ** ((d + 1) ** L) + 1e-12
        # eq:deflated_ns_ratio (gamma^-1 > ell holds here)
        bound = ((1 - phi ** 2) / (1 - ell ** 2)) ** ((d + 1) ** L)
        assert ed <= bound * eb + 1e-12
        if L > 0:
            assert ed < eb


# --- bf16 contract of the filter (ns_step / ns_filter, mode "bf16") --------------
# The contract's rounding points, one step on a stored iterate x:
#   (a) the product operand is hi = bf16(x) (both factors of G, and the right
#       factor of B hi);
#   (b) the iterate is carried as hi + e4m3(clip((x - hi) 2^16)) 2^-16, and
#       the linear term a x takes that carried value;
#   (c) the operand of G^2 is bf16(G) (the linear term b G keeps G wide);
#   (d) B = bf16(b G + c G^2) is the product operand of the update.
# On a diagonal iterate every product is scalar, so each rounding point can be
# checked against a scalar computation that rounds with torch's own bfloat16
# and float8_e4m3fn conversions (a library independent of the oracle's
# rounding code). torch converts float64 through float32, which equals direct
# rounding unless the float32 value lands exactly on a tie of the target
# format; the reference checks that it does not (or that the value is exact
# in float32).
def _torch_round(x, dtype):
    import torch
    x = np.asarray(x, dtype=np.float64)
    x32 = x.astype(np.float32)
    exact = x32.astype(np.float64) == x

    def rnd(v):
        return torch.from_numpy(np.asarray(v, dtype=np.float32)).to(dtype).to(torch.float64).numpy()
    # a float32 value strictly between two ties rounds like its neighbours
    lo = rnd(np.nextafter(x32, np.float32(-np.inf)))
    hi = rnd(np.nextafter(x32, np.float32(np.inf)))
    assert np.all(exact | (lo == hi)), "float32 rounding landed on a tie of the target format"
    return torch.from_numpy(x).to(dtype).to(torch.float64).numpy()


def _scalar_contract_step(x, coeffs, drop=None):
    """One bf16-contract step on the diagonal entries x, with rounding point
    `drop` left out ("a_operand", "b_residual_none", "b_residual_full",
    "c_gram_operand", "d_poly")."""
    import torch
    a, b, c = (float(v) for v in coeffs)
    hi = _torch_round(x, torch.bfloat16)
    res = np.clip((x - hi) * 2.0 ** 16, -448.0, 448.0)
    carried = hi + _torch_round(res, torch.float8_e4m3fn) * 2.0 ** -16
    if drop == "b_residual_none":
        carried = hi
    elif drop == "b_residual_full":
        carried = x
    op = carried if drop == "a_operand" else hi
    g = op * op
    gop = g if drop == "c_gram_operand" else _torch_round(g, torch.bfloat16)
    bw = b * g + c * gop * gop
    bb = bw if drop == "d_poly" else _torch_round(bw, torch.bfloat16)
    return a * carried + bb * op


DROPS = ["a_operand", "b_residual_none", "b_residual_full", "c_gram_operand", "d_poly"]


def test_bf16_contract_step_known_answer_and_each_rounding_point_is_applied():
    # float32 entries whose bf16 residuals are nonzero and inside e4m3's
    # normal range, so every rounding point changes some entry
    x = np.array([0.7, -0.3, 1.05, 0.013, 0.4375, -0.9], dtype=np.float32).astype(np.float64)
    coeffs = (1.875, -1.25, 0.375)       # few-bit coefficients keep the reference float32-exact
    want = _scalar_contract_step(x, coeffs)
    # ns_filter stores the state (a, b) and calls ns_step, which applies (c, d)
    got = ns_filter(np.diag(x), [coeffs], "bf16")
    np.testing.assert_array_equal(np.diag(got), want)
    assert np.count_nonzero(got - np.diag(np.diag(got))) == 0
    for drop in DROPS:
        alt = _scalar_contract_step(x, coeffs, drop)
        assert np.max(np.abs(alt - want)) > 1e-6, f"dropping {drop} left the step unchanged"


def test_bf16_contract_two_steps_muon_coefficients():
    # Muon's quintic (float32 coefficients) over two steps: the second step
    # starts from the stored form of the first one's result
    x = np.array([0.61, -0.27, 0.95, 0.05], dtype=np.float32).astype(np.float64)
    table = np.array([filters.MUON_QUINTIC] * 2, dtype=np.float32).astype(np.float64)
    y1 = _scalar_contract_step(x, table[0])
    np.testing.assert_array_equal(np.diag(ns_filter(np.diag(x), table[:1], "bf16")), y1)
    np.testing.assert_array_equal(np.diag(ns_filter(np.diag(x), table, "bf16")),
                                  _scalar_contract_step(y1, table[1]))


def test_bf16_contract_is_exact_on_dyadic_input():
    # Entries and coefficients on a coarse dyadic grid keep every operand,
    # product and polynomial value exactly representable in bf16 and the
    # state exactly representable as hi plus an e4m3 residual: the contract
    # must then equal exact arithmetic bit for bit (no rounding point rounds
    # to a coarser grid or is applied to a wide value inexactly).
    quintic = np.diag([0.5, -0.25, 1.0, 0.0, -0.5])
    np.testing.assert_array_equal(ns_filter(quintic, [(1.875, -1.25, 0.375)], "bf16"),
                                  ns_filter(quintic, [(1.875, -1.25, 0.375)]))
    cubic = np.diag([1.0, 0.0, -1.0, 0.5, -0.5, 0.75])
    for table in ([(1.5, -0.5, 0.0)], [(1.5, -0.5, 0.0)] * 2):
        if len(table) == 2:
            cubic = cubic[:5, :5]    # 0.75 leaves a 12-bit Gram after one step
        np.testing.assert_array_equal(ns_filter(cubic, table, "bf16"), ns_filter(cubic, table))


def test_bf16_contract_commutes_with_signed_permutations_and_transpose():
    # Every rounding is elementwise, so for X = P D Q^T with signed
    # permutations P, Q the contract gives P f(D) Q^T exactly, on the tall
    # and the wide orientation alike (short-side Gram on both).
    rng = np.random.default_rng(3)
    d = np.array([0.81, -0.33, 0.57, 0.12, 0.98], dtype=np.float32).astype(np.float64)
    table = np.array([filters.MUON_QUINTIC] * 3, dtype=np.float32).astype(np.float64)
    fd = np.diag(ns_filter(np.diag(d), table, "bf16"))
    for rows, cols in ((5, 9), (9, 5)):
        p = np.eye(rows)[rng.permutation(rows)] * rng.choice([-1.0, 1.0], rows)
        q = np.eye(cols)[rng.permutation(cols)] * rng.choice([-1.0, 1.0], cols)
        dd = np.zeros((rows, cols))
        dd[:5, :5] = np.diag(d)
        ff = np.zeros((rows, cols))
        ff[:5, :5] = np.diag(fd)
        np.testing.assert_array_equal(ns_filter(p @ dd @ q.T, table, "bf16"), p @ ff @ q.T)
