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
