"""Seeded synthetic inputs shaped like the paper's workloads.

This module is shared by the tests, the benchmark and the smoke check. It holds
no arithmetic of the method itself: it only draws random spectra and random
orthogonal factors and assembles ``U diag(s) V^T`` (or ``Q diag(lam) Q^T``),
then rounds the result to the storage dtype.

Stand-ins (the paper's data is not available):
  * Muon inputs stand in for recorded GPT-2 momentum matrices (Sec. 3.1 and
    App. D): a few dominant singular values over a log-uniform bulk near zero,
    the head-dominated shape of the paper's momentum spectra (Sec. 2.1).
  * PSD inputs stand in for the ADMM iterates of the Mittelmann max-cut SDPs
    (Sec. 3.3): symmetric matrices with a few dominant eigenvalues of both
    signs over a bulk in [-1, 1].

Every array is a pure function of (MASTER_SEED, workload id, extra ids).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

MASTER_SEED = 21102

# Muon's retuned quintic (Sec. 3 setup); stored as the float32 values the
# library receives.
MUON_COEFFS = (3.4445, -4.7750, 2.0315)


def rng_for(*ids: int) -> np.random.Generator:
    return np.random.default_rng([MASTER_SEED, *[int(i) for i in ids]])


# ---------------------------------------------------------------- storage ---
def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float data to bfloat16 (via float32, round-to-nearest-even).

    Returns the raw 16-bit patterns as uint16. Used only to create inputs.
    """
    f = np.ascontiguousarray(np.asarray(a, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    nan = np.isnan(f)
    out = r.astype(np.uint16)
    if nan.any():
        out[nan] = np.uint16(0x7FC0)
    return out


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    u = np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


# ------------------------------------------------------------ primitives ---
def haar_orthogonal(rng: np.random.Generator, n: int, k: int | None = None) -> np.ndarray:
    """n x k matrix with orthonormal columns from QR of a Gaussian block,
    signs fixed so the distribution is Haar (Mezzadri 2007)."""
    k = n if k is None else k
    g = rng.standard_normal((n, k))
    q, r = np.linalg.qr(g)
    d = np.sign(np.diag(r))
    d[d == 0] = 1.0
    return q * d


def log_uniform(rng: np.random.Generator, lo: float, hi: float, size: int) -> np.ndarray:
    return 10.0 ** rng.uniform(math.log10(lo), math.log10(hi), size=size)


def spiked_matrix(rng, rows, cols, spikes, bulk_lo, bulk_hi):
    """rows x cols matrix U diag(s) V^T (float64) with the given leading
    singular values and a log-uniform bulk; returns (M, s_sorted)."""
    q = min(rows, cols)
    spikes = np.asarray(spikes, dtype=np.float64)
    bulk = log_uniform(rng, bulk_lo, bulk_hi, q - spikes.size)
    s = np.concatenate([spikes, bulk])
    u = haar_orthogonal(rng, rows, q)
    v = haar_orthogonal(rng, cols, q)
    m = (u * s) @ v.T
    return m, np.sort(s)[::-1]


def symmetric_from_spectrum(rng, lam):
    n = lam.size
    q = haar_orthogonal(rng, n)
    z = (q * lam) @ q.T
    z = 0.5 * (z + z.T)
    return z, q


# --------------------------------------------------------------- Muon ------
@dataclass
class MuonCase:
    name: str
    x: np.ndarray              # [B, m, n]: float32 array, or uint16 bf16 bits
    dtype: str                 # "f32" | "bf16"
    k: int
    oversample: int
    power_iters: int
    steps: int
    coeffs: np.ndarray         # float32 [steps, 3]
    gamma: float
    spectra: list = field(default_factory=list)   # true singular values (f64)

    @property
    def x64(self) -> np.ndarray:
        if self.dtype == "bf16":
            return bf16_bits_to_f64(self.x)
        return self.x.astype(np.float64)


def muon_coeff_table(steps: int) -> np.ndarray:
    return np.tile(np.asarray(MUON_COEFFS, dtype=np.float32), (steps, 1))


def polar_express_like_table(seed_id: int, steps: int = 8) -> np.ndarray:
    """A seeded per-step table of degree-5 odd polynomial coefficients.

    The paper's Polar-Express coefficients are not printed, so the table is a
    bounded family between Muon's quintic and the classical one (15/8, -5/4,
    3/8) with a small seeded jitter, stored as float32 [steps, 3].
    """
    rng = rng_for(903, seed_id)
    muon = np.asarray(MUON_COEFFS, dtype=np.float64)
    classical = np.array([15 / 8, -5 / 4, 3 / 8])
    rows = []
    for t in range(steps):
        w = t / max(steps - 1, 1)
        base = (1 - w) * muon + w * classical
        jitter = 1.0 + 0.02 * rng.uniform(-1.0, 1.0, size=3)
        rows.append(base * jitter)
    return np.asarray(rows, dtype=np.float32)


def muon_batch(name, batch, m, n, *, dtype, spikes, bulk, k, oversample,
               power_iters, steps, coeffs, gamma, ids) -> MuonCase:
    xs, spectra = [], []
    for b in range(batch):
        rng = rng_for(*ids, b)
        mat, s = spiked_matrix(rng, m, n, spikes, bulk[0], bulk[1])
        xs.append(mat)
        spectra.append(s)
    x = np.stack(xs)
    if dtype == "bf16":
        x = to_bf16_bits(x)
    else:
        x = x.astype(np.float32)
    return MuonCase(name, x, dtype, k, oversample, power_iters, steps,
                    np.asarray(coeffs, dtype=np.float32), gamma, spectra)


def config1() -> MuonCase:
    """One fp32 256 x 256 matrix: spikes 100 * 2^-i (i = 0..3) over a
    log-uniform bulk in [1e-3, 1]; k = 4, oversample 8, 2 power iterations,
    5 steps of Muon's quintic."""
    spikes = [100.0 * 2.0 ** -i for i in range(4)]
    return muon_batch("c1_256x256_f32", 1, 256, 256, dtype="f32", spikes=spikes,
                      bulk=(1e-3, 1.0), k=4, oversample=8, power_iters=2, steps=5,
                      coeffs=muon_coeff_table(5), gamma=1.01, ids=(1,))


C2_GROUPS = {"768x768": (12, 768, 768), "768x2304": (12, 768, 2304),
             "768x3072": (24, 768, 3072)}


def config2(group: str = "768x3072", batch: int | None = None) -> MuonCase:
    """GPT-2-small-shaped bf16 Muon batch: 8 spikes geometric from 50 down to
    5 over a log-uniform bulk in [1e-4, 1]; k = 8, oversample 8, 1 power
    iteration, 5 steps of Muon's quintic."""
    b, m, n = C2_GROUPS[group]
    b = b if batch is None else batch
    spikes = [50.0 * 10.0 ** (-i / 7.0) for i in range(8)]
    gid = list(C2_GROUPS).index(group)
    return muon_batch(f"c2_{b}x{group}_bf16", b, m, n, dtype="bf16", spikes=spikes,
                      bulk=(1e-4, 1.0), k=8, oversample=8, power_iters=1, steps=5,
                      coeffs=muon_coeff_table(5), gamma=1.01, ids=(2, gid))


def config3(group: str = "768x3072", batch: int | None = None) -> MuonCase:
    """Config-2 shapes and spectra with a seeded 8 x 3 Polar-Express-style
    table, k = 16, gamma = 1.1."""
    c = config2(group, batch)
    c.name = c.name.replace("c2_", "c3_")
    c.k = 16
    c.steps = 8
    c.coeffs = polar_express_like_table(0, 8)
    c.gamma = 1.1
    return c


# The paper's GPT-2 Large Muon groups (App. D): 144 square 1280 x 1280 and 72
# tall 5120 x 1280 matrices, deflation rank 32 with 64 sketch columns.
PAPER_GROUPS = {"1280x1280": (144, 1280, 1280), "5120x1280": (72, 5120, 1280)}


def paper_scale_group(group: str, distinct: int = 6) -> MuonCase:
    """A paper-scale bf16 group: 32 spikes geometric from 50 down to 5 over a
    log-uniform bulk in [1e-4, 1]; k = 32, oversample 32 (r' = 64), 1 power
    iteration, 5 steps of Muon's quintic. The batch cycles through `distinct`
    seeded matrices (matrix b is matrix b mod distinct); every batch position
    still draws its own sketch, so each position is an independent case."""
    b, m, n = PAPER_GROUPS[group]
    spikes = [50.0 * 10.0 ** (-i / 31.0) for i in range(32)]
    gid = list(PAPER_GROUPS).index(group)
    pool = muon_batch(f"paper_{group}_pool", distinct, m, n, dtype="bf16", spikes=spikes,
                      bulk=(1e-4, 1.0), k=32, oversample=32, power_iters=1, steps=5,
                      coeffs=muon_coeff_table(5), gamma=1.01, ids=(6, gid))
    idx = np.arange(b) % distinct
    pool.name = f"paper_{b}x{group}_bf16"
    pool.x = np.ascontiguousarray(pool.x[idx])
    pool.spectra = [pool.spectra[i] for i in idx]
    return pool


def small_muon(b, m, n, *, dtype="f32", k=4, spikes=None, bulk=(1e-3, 1.0),
               oversample=8, power_iters=1, steps=5, coeffs=None, gamma=1.01,
               case_id=0) -> MuonCase:
    """Small spiked cases for parity sweeps (ragged shapes, tall and wide)."""
    q = min(m, n)
    if spikes is None:
        nsp = min(max(k, 1), q)
        spikes = [50.0 * 10.0 ** (-i / 7.0) for i in range(nsp)]
    spikes = list(spikes)[:q]
    coeffs = muon_coeff_table(steps) if coeffs is None else coeffs
    return muon_batch(f"small_{b}x{m}x{n}_{dtype}_k{k}", b, m, n, dtype=dtype,
                      spikes=spikes, bulk=bulk, k=k, oversample=oversample,
                      power_iters=power_iters, steps=steps, coeffs=coeffs,
                      gamma=gamma, ids=(100, case_id, m, n, k))


# ---------------------------------------------------------------- PSD ------
@dataclass
class PSDCase:
    name: str
    z: np.ndarray            # float32 [n, n], exactly symmetric
    lam: np.ndarray          # eigenvalues (f64) the matrix was built from
    q: np.ndarray | None     # eigenvectors (f64), or None when not kept
    k: int
    subspace_iters: int
    steps: int
    gamma: float
    qwarm: np.ndarray        # float32 [n, k] warm-start basis


def psd_spectrum(rng, n, n_dom, dom_lo, dom_hi):
    mags = rng.uniform(dom_lo, dom_hi, size=n_dom)
    while True:
        signs = np.where(rng.uniform(size=n_dom) < 0.5, -1.0, 1.0)
        if n_dom < 2 or (signs > 0).any() and (signs < 0).any():
            break
    bulk = rng.uniform(-1.0, 1.0, size=n - n_dom)
    return np.concatenate([mags * signs, bulk])


def warm_basis(rng, q_top, eps):
    """Orthonormalized seeded perturbation of the true top eigenvectors."""
    n, k = q_top.shape
    g = rng.standard_normal((n, k))
    w = q_top + eps * g / math.sqrt(n)
    qq, r = np.linalg.qr(w)
    return qq * np.sign(np.diag(r))


def psd_case(name, n, n_dom, dom, k, subspace_iters, steps, gamma, ids,
             eps=1e-2) -> PSDCase:
    rng = rng_for(*ids)
    lam = psd_spectrum(rng, n, n_dom, dom[0], dom[1])
    z, q = symmetric_from_spectrum(rng, lam)
    order = np.argsort(-np.abs(lam), kind="stable")
    qw = warm_basis(rng, q[:, order[:k]], eps)
    z32 = z.astype(np.float32)
    z32 = np.triu(z32) + np.triu(z32, 1).T     # exactly symmetric storage
    return PSDCase(name, z32, lam, q, k, subspace_iters, steps, gamma,
                   qw.astype(np.float32))


def config4() -> PSDCase:
    """n = 4096 fp32: 10 dominant eigenvalues +-U[200, 1000] over a bulk
    U[-1, 1]; k = 16, warm start at eps = 1e-2, 2 subspace iterations,
    10 cubic Newton-Schulz sign steps."""
    return psd_case("c4_4096_f32", 4096, 10, (200.0, 1000.0), 16, 2, 10, 1.1, ids=(4,))


def small_psd(n, *, k=8, n_dom=4, dom=(50.0, 200.0), subspace_iters=2, steps=10,
              gamma=1.1, case_id=0, eps=1e-2) -> PSDCase:
    return psd_case(f"psd_small_{n}_k{k}", n, n_dom, dom, k, subspace_iters, steps,
                    gamma, ids=(200, case_id, n, k), eps=eps)


def low_rank(b: int, m: int, n: int, rank: int, case_id: int = 0) -> np.ndarray:
    """float32 [b, m, n] of exact rank `rank` (U diag(s) V^T, s = 10, 5, ...,
    U and V orthonormal from Gaussian QR): a degenerate input whose sketch
    panels are rank-deficient once the sketch is wider than the rank."""
    rng = rng_for(700, case_id, m, n, rank)
    out = np.empty((b, m, n), dtype=np.float32)
    for i in range(b):
        u, _ = np.linalg.qr(rng.standard_normal((m, rank)))
        v, _ = np.linalg.qr(rng.standard_normal((n, rank)))
        sv = 10.0 * 0.5 ** np.arange(rank)
        out[i] = ((u * sv) @ v.T).astype(np.float32)
    return out


def sym_gaussian(n: int, case_id: int = 0) -> np.ndarray:
    """Seeded symmetric Gaussian matrix (G + G^T) / sqrt(2), float32, exactly
    symmetric (a semicircle spectrum of radius about 2 sqrt(n))."""
    g = rng_for(600, case_id, n).standard_normal((n, n)).astype(np.float32)
    z = (g + g.T) / np.float32(math.sqrt(2.0))
    return np.triu(z) + np.triu(z, 1).T


def psd_drift(z: np.ndarray, rel: float, call: int, case_id: int = 5) -> np.ndarray:
    """Seeded symmetric perturbation E with ||E||_F = rel * ||Z||_F."""
    rng = rng_for(500, case_id, call)
    n = z.shape[0]
    g = rng.standard_normal((n, n)).astype(np.float32)
    e = (g + g.T) / math.sqrt(2.0)
    e *= np.float32(rel * np.linalg.norm(z) / np.linalg.norm(e))
    out = (z + e).astype(np.float32)
    return np.triu(out) + np.triu(out, 1).T


def config5_first(n: int = 16384) -> PSDCase:
    """n = 16384 fp32: 32 dominant eigenvalues +-U[500, 5000] over a bulk
    U[-1, 1]; k = 32, one subspace iteration per call, 10 cubic steps.

    Building it needs an n x n QR (minutes of host time at n = 16384)."""
    return psd_case(f"c5_{n}_f32", n, 32, (500.0, 5000.0), 32, 1, 10, 1.1, ids=(5,))


def config5_device(n: int = 16384, device: str = "cuda"):
    """Config 5 at full size, assembled on the GPU.

    Same recipe as config5_first (32 dominant eigenvalues +-U[500, 5000] over
    a bulk U[-1, 1], warm start at eps = 1e-2), drawn from the same seeded
    host generator, but the n x n orthogonal factor comes from a float64
    Householder QR on the GPU and Q diag(lam) Q^T from a float64 product
    there: at n = 16384 the host QR takes minutes. Returns (z, lam, q, qwarm):
    z float32 [n, n] exactly symmetric, lam float64 numpy [n], q float64
    [n, n] (device), qwarm float32 [n, 32] (device)."""
    import torch
    rng = rng_for(5)
    lam = psd_spectrum(rng, n, 32, 500.0, 5000.0)
    g = torch.from_numpy(rng.standard_normal((n, n))).to(device)
    q, r = torch.linalg.qr(g)
    del g
    q *= torch.sign(torch.diagonal(r)).unsqueeze(0)
    del r
    lam_d = torch.from_numpy(lam).to(device)
    z64 = (q * lam_d) @ q.T
    z64 = 0.5 * (z64 + z64.T)
    z = z64.float()
    del z64
    z = torch.triu(z) + torch.triu(z, 1).T   # exactly symmetric storage
    order = np.argsort(-np.abs(lam), kind="stable")
    top = q[:, torch.from_numpy(order[:32]).to(device)]
    w = top + 1e-2 * torch.from_numpy(rng.standard_normal((n, 32))).to(device) / math.sqrt(n)
    qq, rr = torch.linalg.qr(w)
    qwarm = (qq * torch.sign(torch.diagonal(rr)).unsqueeze(0)).float().contiguous()
    return z.contiguous(), lam, q, qwarm


def psd_drift_device(z, rel: float, call: int, case_id: int = 5):
    """psd_drift on the GPU: E = (G + G^T) / sqrt(2) from a seeded device
    generator, scaled to ||E||_F = rel ||Z||_F; z + E stored exactly
    symmetric (float32)."""
    import torch
    gen = torch.Generator(device=z.device)
    gen.manual_seed(MASTER_SEED * 1000003 + case_id * 1009 + call)
    n = z.shape[0]
    e = torch.randn((n, n), generator=gen, device=z.device, dtype=torch.float32)
    e = (e + e.T) / math.sqrt(2.0)
    e *= (rel * torch.linalg.norm(z.double()) / torch.linalg.norm(e.double())).float()
    out = z + e
    return (torch.triu(out) + torch.triu(out, 1).T).contiguous()


# ----------------------------------------------------------------- ADMM -----
@dataclass
class MaxCutCase:
    name: str
    w: np.ndarray            # symmetric 0/1 weights, zero diagonal (float64)
    c: np.ndarray            # cost -L / 4 of the relaxation min <C, X>, diag(X) = 1 (float32)
    b: np.ndarray            # ones (float32)
    basis0: np.ndarray       # float32 [n, K]: orthonormalized Gaussian start of the tracked basis
    k: int                   # K = ceil(0.05 n) tracked columns (Sec. 3.3: w' = 0.05)
    window: int              # r = ceil(0.025 n) (w = 0.025)


def planted_maxcut(n: int, case_id: int = 0, p_in: float = 0.01, p_out: float = 0.15) -> MaxCutCase:
    """Max-cut relaxation of a random graph with a planted bisection (edges
    across the two halves with probability p_out, inside with p_in): a
    stand-in for the Gset max-cut instances of the paper's SDP runs (Sec. 3.3),
    whose ADMM iterates have a dominant head over a bulk."""
    rng = rng_for(7, case_id, n)
    lab = np.arange(n) % 2
    prob = np.where(lab[:, None] == lab[None, :], p_in, p_out)
    a = np.triu((rng.uniform(size=(n, n)) < prob).astype(np.float64), 1)
    w = a + a.T
    lap = np.diag(w.sum(axis=1)) - w
    c = (-0.25 * lap).astype(np.float32)
    k = math.ceil(0.05 * n)
    g = rng.standard_normal((n, k))
    q, r = np.linalg.qr(g)
    basis0 = (q * np.sign(np.diag(r))).astype(np.float32)
    return MaxCutCase(f"maxcut_planted_{n}", w, c, np.ones(n, dtype=np.float32), basis0, k,
                      math.ceil(0.025 * n))

