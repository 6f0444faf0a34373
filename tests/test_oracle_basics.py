"""Pins of oracle.precision, oracle.rng and oracle.linalg."""
import numpy as np
import pytest
import torch
from scipy import stats

from oracle import linalg, precision, rng


# --- bf16 rounding ---------------------------------------------------------------
def test_bf16_ties_and_exact_values():
    r = precision.round_bf16
    one = 1.0
    assert r(np.array([one]))[0] == 1.0
    assert r(np.array([1 + 2.0 ** -8]))[0] == 1.0                       # tie -> even
    assert r(np.array([1 + 3 * 2.0 ** -8]))[0] == 1 + 2.0 ** -6         # tie -> even
    assert r(np.array([-(1 + 3 * 2.0 ** -8)]))[0] == -(1 + 2.0 ** -6)
    assert r(np.array([1 + 2.0 ** -8 + 2.0 ** -30]))[0] == 1 + 2.0 ** -7  # above tie
    assert r(np.array([0.0]))[0] == 0.0


def test_bf16_matches_library_rounding():
    # Values that are exact in float32 round the same as torch's float32 -> bfloat16.
    g = np.random.default_rng(0)
    x = (g.standard_normal(200000) * 10.0 ** g.uniform(-6, 6, 200000)).astype(np.float32)
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(precision.round_bf16(x.astype(np.float64)), want)


# --- fp16 rounding (operands of the fp16 sign filter) ---------------------------
def test_f16_ties_subnormals_and_exact_values():
    r = precision.round_f16
    assert r(np.array([1 + 2.0 ** -11]))[0] == 1.0                        # tie -> even
    assert r(np.array([1 + 3 * 2.0 ** -11]))[0] == 1 + 2.0 ** -9          # tie -> even
    assert r(np.array([-(1 + 2.0 ** -11 + 2.0 ** -40)]))[0] == -(1 + 2.0 ** -10)
    assert r(np.array([2.0 ** -24]))[0] == 2.0 ** -24                     # smallest subnormal
    assert r(np.array([2.0 ** -25]))[0] == 0.0                            # tie -> even (zero)
    assert r(np.array([3 * 2.0 ** -25]))[0] == 2.0 ** -23                 # tie -> even
    assert r(np.array([65504.0]))[0] == 65504.0
    with pytest.raises(ValueError):
        r(np.array([65505.0]))


def test_f16_matches_library_rounding():
    g = np.random.default_rng(5)
    x = (g.standard_normal(200000) * 10.0 ** g.uniform(-9, 4, 200000)).astype(np.float32)
    x = np.clip(x, -65504, 65504)
    want = torch.from_numpy(x).to(torch.float16).to(torch.float64).numpy()
    np.testing.assert_array_equal(precision.round_f16(x.astype(np.float64)), want)


# --- e4m3 rounding (residual of the stored bf16 iterate) -------------------------
def _e4m3_grid():
    """Every finite OCP e4m3 ("fn") value from its bit layout: sign, 4-bit
    exponent field (bias 7), 3-bit fraction; field 0 is subnormal, field 15
    with fraction 7 is NaN."""
    vals, codes = [], []
    for b in range(256):
        e, m = (b >> 3) & 0xF, b & 7
        if e == 0xF and m == 7:
            continue
        v = (m / 8) * 2.0 ** -6 if e == 0 else (1 + m / 8) * 2.0 ** (e - 7)
        vals.append(-v if b & 0x80 else v)
        codes.append(b)
    return np.array(vals), np.array(codes)


def test_e4m3_matches_nearest_grid_value():
    grid, codes = _e4m3_grid()
    assert grid.max() == 448.0 and np.sort(np.abs(grid))[2] == 2.0 ** -9
    g = np.random.default_rng(3)
    pos = np.unique(np.abs(grid))
    mids = (pos[1:] + pos[:-1]) / 2
    x = np.concatenate([g.uniform(-448, 448, 20000), g.standard_normal(20000) * 10.0 ** g.uniform(-4, 2, 20000),
                        mids, -mids, np.nextafter(mids, 0), np.nextafter(mids, 1e9), pos, -pos])
    x = np.clip(x, -448, 448)
    d = np.abs(x[:, None] - grid[None, :])
    best = d.min(axis=1, keepdims=True)
    tie_ok = (d == best)
    # ties go to the even fraction (lowest code bit clear)
    pick = np.where(tie_ok & ((codes[None, :] & 1) == 0), 1, 0) + np.where(tie_ok, 1, 0)
    want = grid[np.argmax(pick, axis=1)]
    got = precision.round_e4m3(x)
    np.testing.assert_array_equal(np.abs(got), np.abs(want))
    assert np.all((got == 0) | (np.sign(got) == np.sign(x)))


def test_e4m3_matches_library_rounding():
    g = np.random.default_rng(4)
    x = np.clip(g.standard_normal(100000) * 10.0 ** g.uniform(-4, 2.5, 100000), -448, 448).astype(np.float32)
    want = torch.from_numpy(x).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    np.testing.assert_array_equal(precision.round_e4m3(x.astype(np.float64)), want)
    with pytest.raises(ValueError):
        precision.round_e4m3(np.array([449.0]))


def test_stored_state_residual():
    from oracle.filters import STATE_SCALE, store_state
    g = np.random.default_rng(5)
    x = g.standard_normal(50000) * 10.0 ** g.uniform(-3, 0.2, 50000)
    hi, carried = store_state(x)
    np.testing.assert_array_equal(hi, precision.round_bf16(x))
    r = (carried - hi) * STATE_SCALE
    # the residual is an e4m3 value, within half a unit in its 4th bit of (x - hi) 2^16
    grid, _ = _e4m3_grid()
    assert np.isin(r, grid).all()
    d = (x - hi) * STATE_SCALE
    inside = np.abs(d) <= 448
    normal = inside & (np.abs(d) >= 2.0 ** -6)
    assert np.all(np.abs(r - d)[normal] <= np.abs(d)[normal] * 2.0 ** -4 * (1 + 1e-12))
    assert np.all(np.abs(r - d)[np.abs(d) < 2.0 ** -6] <= 2.0 ** -10)
    np.testing.assert_array_equal(r[~inside], np.sign(d[~inside]) * 448.0)
    assert inside.mean() > 0.9
    # round trip: an iterate already in stored form keeps its value (and its
    # split, unless the residual rounded to half a bf16 unit, a tie of bf16)
    hi2, carried2 = store_state(carried)
    np.testing.assert_array_equal(carried2, carried)
    half_ulp = np.abs(hi) * 2.0 ** -8   # at or above half a unit of hi
    split_kept = np.abs(carried - hi) < np.ldexp(1.0, np.frexp(hi)[1] - 9)
    assert split_kept.mean() > 0.9 and np.all(np.abs(carried - hi) <= half_ulp + 1e-300)
    np.testing.assert_array_equal(hi2[split_kept], hi[split_kept])
    # residuals past the format's range are clipped to +-448 2^-16
    big = np.array([3.0 + 0.45 * 2.0 ** -6, -(3.0 + 0.45 * 2.0 ** -6)])   # residual 0.45 units of 2^-6
    hb, cb = store_state(big)
    np.testing.assert_array_equal(cb - hb, np.sign(big) * 448.0 / STATE_SCALE)


# --- Gaussian generator ------------------------------------------------------------
# Known-answer vectors of Philox4x32-10 published with the generator
# (Salmon, Moraes, Dror, Shaw, SC 2011; Random123 distribution): counter,
# key -> output, all words as 32-bit integers.
PHILOX_KAT = [
    ((0x00000000, 0x00000000, 0x00000000, 0x00000000), (0x00000000, 0x00000000),
     (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF), (0xFFFFFFFF, 0xFFFFFFFF),
     (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
]


@pytest.mark.parametrize("ctr,key,want", PHILOX_KAT)
def test_philox_known_answers(ctr, key, want):
    args = [np.array([v], dtype=np.uint32) for v in (*ctr, *key)]
    got = [int(np.asarray(w).ravel()[0]) for w in rng.philox4x32_10(*args)]
    assert got == list(want)


def test_gaussians_are_standard_normal():
    z = rng.gaussians(0, 0, rng.STREAM_SKETCH, 200000)
    assert abs(z.mean()) < 0.01 and abs(z.var() - 1) < 0.01
    assert stats.kstest(z, "norm").pvalue > 1e-3


def test_streams_and_matrices_independent():
    a = rng.gaussians(0, 0, 1, 50000)
    b = rng.gaussians(0, 1, 1, 50000)
    c = rng.gaussians(0, 0, 2, 50000)
    d = rng.gaussians(1, 0, 1, 50000)
    for other in (b, c, d):
        assert abs(np.corrcoef(a, other)[0, 1]) < 0.02
    # lanes within one call are not correlated either
    lanes = a[:48000].reshape(-1, 4)
    cc = np.corrcoef(lanes.T)
    assert np.all(np.abs(cc - np.eye(4)) < 0.03)


def test_gaussians_prefix_stable_and_float32():
    a = rng.gaussians(5, 3, 1, 1001)
    b = rng.gaussians(5, 3, 1, 37)
    np.testing.assert_array_equal(a[:37], b)
    assert np.all(a.astype(np.float32).astype(np.float64) == a)


def test_sketch_layout_is_column_major():
    om = rng.sketch(9, 2, 13, 5)
    g = rng.gaussians(9, 2, rng.STREAM_SKETCH, 65)
    assert om.shape == (13, 5)
    assert om[4, 3] == g[3 * 13 + 4]


# --- CholeskyQR --------------------------------------------------------------------
@pytest.mark.parametrize("cond", [1.0, 1e2, 1e4])
def test_cholqr_orthonormal_and_same_span(cond):
    g = np.random.default_rng(1)
    n, c = 500, 12
    u, _ = np.linalg.qr(g.standard_normal((n, c)))
    w, _ = np.linalg.qr(g.standard_normal((c, c)))
    p = (u * np.logspace(0, -np.log10(cond), c)) @ w
    q = linalg.cholqr(p)
    # one pass: orthogonality error about kappa^2 u
    np.testing.assert_allclose(q.T @ q, np.eye(c), atol=100 * cond ** 2 * 2.0 ** -53 + 1e-13)
    qn, _ = np.linalg.qr(p)                                      # library Householder QR
    np.testing.assert_allclose(q @ np.linalg.pinv(q), qn @ qn.T, atol=1e-9)
    # R = Q^+ P is upper triangular with a positive diagonal
    r = np.linalg.pinv(q) @ p
    assert np.allclose(np.tril(r, -1), 0, atol=1e-9 * np.abs(r).max())
    assert np.all(np.diag(r) > 0)


def test_cholqr_degenerate_panels():
    z = np.zeros((40, 4))
    np.testing.assert_array_equal(linalg.cholqr(z), z)
    g = np.random.default_rng(2)
    p = g.standard_normal((40, 2)) @ g.standard_normal((2, 4))   # rank 2 of 4
    q = linalg.cholqr(p)
    assert np.all(np.isfinite(q))
    # the first two columns span range(P) and are orthonormal; the floored
    # pivots leave the dependent columns small
    np.testing.assert_allclose(q[:, :2].T @ q[:, :2], np.eye(2), atol=1e-12)
    np.testing.assert_allclose(q[:, :2] @ (q[:, :2].T @ p), p, atol=1e-10 * np.abs(p).max())
    assert np.linalg.norm(q[:, 2:]) < 1e-4


def test_cholesky_upper_matches_library():
    g = np.random.default_rng(3)
    a = g.standard_normal((30, 9))
    gram = a.T @ a
    r = linalg.cholesky_upper(gram, 0.0)
    np.testing.assert_allclose(r, np.linalg.cholesky(gram).T, rtol=1e-12, atol=1e-12)
