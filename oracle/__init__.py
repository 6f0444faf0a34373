"""CPU oracle for the spectrally deflated polynomial filters.

TEST INFRASTRUCTURE ONLY. This package is a plain, slow, float64 NumPy
implementation of what the GPU library computes, written from the paper
(arXiv 2609.21102, "Spectral Deflation for Factorization-Free Matrix Filtering
in Muon and Semidefinite Programming"). Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import it. It shares no code, headers, tables
or helpers with the HIP library, and the library never calls it.

Modules
  rng        Philox4x32-10 counter generator and the Box-Muller transform that
             produce the Gaussian sketch and the Lanczos start vector.
  precision  bfloat16 round-to-nearest-even, used by the "bf16" contract mode.
  filters    Newton-Schulz family: Bjorck-Bowie coefficients (App. B), the
             scalar odd polynomials and one matrix step (eq:muon_ns,
             eq:general_ns_iteration).
  linalg     CholeskyQR of a tall panel.
  muon       Batched randomized SVD (Alg. 3), the deflated polar factor
             (Alg. 1), the undeflated baseline and the exact polar factor.
  psd        Lanczos scale estimate (App. E.1), the deflated PSD projection
             (Alg. 2), the undeflated baseline (eq:baseline_projection) and the
             exact projection (eq:psd_sign).
  admm       Three-block ADMM for SDPs with diagonal constraints (the max-cut
             relaxation; eq:admm_iter) and its KKT residual (eq:admm_eta).

Pins: every function is checked in tests/test_oracle_*.py against values the
paper prints, closed forms, invariants or brute force; none is "parity
unpinned".
"""
from . import admm, filters, linalg, muon, precision, psd, rng  # noqa: F401
