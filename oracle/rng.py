"""Counter-based Gaussian numbers for the sketch and the Lanczos start vector.

The paper draws a Gaussian sketch (Alg. 3, "Omega <- Gaussian(B, m, r')") and
starts Lanczos from a random vector (App. E.1) without fixing a generator.
Both sides of the parity tests therefore implement one published generator:

* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy
  as 1, 2, 3", SC 2011): a 4 x 32-bit counter and a 2 x 32-bit key; each round
  multiplies counter words 0 and 2 by 0xD2511F53 and 0xCD9E8D57, splits the
  64-bit products into high and low halves, xors the high halves with the
  other counter words and the key, and permutes; the key is advanced by the
  Weyl constants 0x9E3779B9, 0xBB67AE85 between rounds; 10 rounds.
* Box-Muller (Box and Muller 1958): two uniforms u1 in (0, 1], u2 in [0, 1)
  give sqrt(-2 ln u1) * (cos 2 pi u2, sin 2 pi u2). A uniform takes the top
  24 bits of a Philox word: u1 = (w >> 8 + 1) / 2^24, u2 = (w >> 8) / 2^24.
  Evaluated in float64, then rounded to float32.

Stream layout (the library uses the same):
  key     = (seed & 0xffffffff, seed >> 32)
  counter = (call, matrix, stream, 0); one call yields 4 Gaussians, so
            Gaussian number g of a (matrix, stream) pair is lane g % 4 of call
            g // 4.
  stream 1: the sketch Omega of one matrix, an (m x r') array filled column by
            column: entry (i, j) is Gaussian number j * m + i.
  stream 2: the Lanczos start vector, entry i is Gaussian number i.
"""
from __future__ import annotations

import numpy as np

_MASK = np.uint64(0xFFFFFFFF)
_M0 = np.uint64(0xD2511F53)
_M1 = np.uint64(0xCD9E8D57)
_W0 = np.uint64(0x9E3779B9)
_W1 = np.uint64(0xBB67AE85)

STREAM_SKETCH = 1
STREAM_LANCZOS = 2


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Vectorised Philox4x32-10. Counter words are arrays (broadcast), key
    words scalars. Returns four uint64 arrays holding 32-bit values."""
    c = [np.asarray(x, dtype=np.uint64) & _MASK for x in (c0, c1, c2, c3)]
    k0 = np.uint64(k0) & _MASK
    k1 = np.uint64(k1) & _MASK
    for _ in range(10):
        p0 = _M0 * c[0]
        p1 = _M1 * c[2]
        hi0, lo0 = p0 >> np.uint64(32), p0 & _MASK
        hi1, lo1 = p1 >> np.uint64(32), p1 & _MASK
        c = [(hi1 ^ c[1] ^ k0) & _MASK, lo1, (hi0 ^ c[3] ^ k1) & _MASK, lo0]
        k0 = (k0 + _W0) & _MASK
        k1 = (k1 + _W1) & _MASK
    return c


def gaussians(seed: int, matrix: int, stream: int, count: int) -> np.ndarray:
    """The first `count` Gaussians of one (matrix, stream) pair, as float64
    holding float32-rounded values."""
    ncall = (count + 3) // 4
    calls = np.arange(ncall, dtype=np.uint64)
    w = philox4x32_10(calls, matrix, stream, 0, seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)
    out = np.empty((ncall, 4), dtype=np.float64)
    scale = 2.0 ** -24
    for pair in range(2):
        a = w[2 * pair].astype(np.float64)
        b = w[2 * pair + 1].astype(np.float64)
        u1 = (np.floor(a / 256.0) + 1.0) * scale
        u2 = np.floor(b / 256.0) * scale
        rad = np.sqrt(-2.0 * np.log(u1))
        ang = 2.0 * np.pi * u2
        out[:, 2 * pair] = rad * np.cos(ang)
        out[:, 2 * pair + 1] = rad * np.sin(ang)
    return out.reshape(-1)[:count].astype(np.float32).astype(np.float64)


def sketch(seed: int, matrix: int, m: int, rprime: int) -> np.ndarray:
    """Omega (m x r') for one matrix of the batch (Alg. 3)."""
    g = gaussians(seed, matrix, STREAM_SKETCH, m * rprime)
    return g.reshape(rprime, m).T.copy()


def lanczos_start(seed: int, n: int) -> np.ndarray:
    """Unnormalised Gaussian start vector for the Lanczos scale estimate."""
    return gaussians(seed, 0, STREAM_LANCZOS, n)
