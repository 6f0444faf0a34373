"""Newton-Schulz family of odd polynomial filters.

* One step of the degree-(2d+1) map (eq:general_ns_iteration; the quintic of
  eq:muon_ns is d = 2):  N(X) = sum_i a_i (X X^T)^i X.
  Since (X X^T)^i X = X (X^T X)^i, the step is evaluated with the Gram matrix
  of the short side (the two forms are equal in exact arithmetic):
      G = X^T X (tall X) or X X^T (wide X),
      B = sum_{i>=1} a_i G^i,
      N(X) = a_0 X + X B (tall) or a_0 X + B X (wide).
* On singular values the step applies p(x) = sum_i a_i x^(2i+1) (Sec. 2.1).
* Bjorck-Bowie coefficients (App. B):
      a_i = (-1)^i sum_{j=i..d} 4^-j C(2j, j) C(j, i).
* Muon's retuned quintic (Sec. 3 setup): (3.4445, -4.7750, 2.0315).

bf16 contract (mode "bf16"), used for the bf16 library paths ("bfloat16
mixed precision" of Sec. 3: bf16 operands, wider accumulation and state): the
iterate is stored as hi = bf16(X) plus a one-byte residual, the float8 e4m3
value r = e4m3(clip((X - hi) 2^16, -448, 448)) (round to nearest even), and
carried as hi + r 2^-16 (the residual keeps 4 significant bits of X - hi, so
the carried value has about 12 or more significant bits where
2^-13 <= |X| < 2; smaller entries keep 4 bits of their residual down to the
format's subnormal range, larger ones a clipped residual);
every matrix product takes bf16 operands, the iterate's being hi, so
G = hi^T hi; the operand of G^2 is bf16(G); B = bf16(b G + c G^2) (with the
unrounded G) is a product operand; the new iterate a (carried X) + hi B is
stored in the same form before the next step. ns_filter returns the last
step's value as computed; the caller rounds it to its output precision.

fp16 contract (mode "f16"), used for the PSD sign filter in fp16 (the paper's
SDP experiments run the filter in fp16, App. E): every product operand is
rounded to fp16 (X for G = X X, G for G^2, and B = b G + c G^2), the products
accumulate wide, and the iterate is stored wide.
"""
from __future__ import annotations

from fractions import Fraction
from math import comb

import numpy as np

from .precision import E4M3_MAX, round_bf16, round_e4m3, rounding

STATE_SCALE = 2.0 ** 16   # residual scale of the stored bf16-contract iterate

MUON_QUINTIC = (3.4445, -4.7750, 2.0315)


def bjorck_bowie(d: int) -> list[Fraction]:
    """Coefficients a_0..a_d of the classical degree-(2d+1) map (App. B)."""
    if d < 1:
        raise ValueError("d >= 1")
    out = []
    for i in range(d + 1):
        acc = Fraction(0)
        for j in range(i, d + 1):
            acc += Fraction(comb(2 * j, j) * comb(j, i), 4 ** j)
        out.append(acc if i % 2 == 0 else -acc)
    return out


def scalar_poly(x, coeffs) -> np.ndarray:
    """p(x) = sum_i coeffs[i] x^(2i+1)."""
    x = np.asarray(x, dtype=np.float64)
    x2 = x * x
    acc = np.zeros_like(x)
    for c in reversed(list(coeffs)):
        acc = acc * x2 + float(c)
    return acc * x


def scalar_compose(x, table) -> np.ndarray:
    """p_L o ... o p_1 (x) for a per-step coefficient table."""
    y = np.asarray(x, dtype=np.float64)
    for row in table:
        y = scalar_poly(y, row)
    return y


def store_state(x: np.ndarray):
    """The stored form of a bf16-contract iterate: returns (hi, carried) with
    hi = bf16(x) and carried = hi + r 2^-16 for the e4m3 residual
    r = e4m3(clip((x - hi) 2^16, -448, 448))."""
    x = np.asarray(x, dtype=np.float64)
    hi = round_bf16(x)
    r = round_e4m3(np.clip((x - hi) * STATE_SCALE, -E4M3_MAX, E4M3_MAX))
    return hi, hi + r / STATE_SCALE


def ns_step(x: np.ndarray, coeffs, mode: str = "exact", operand=None) -> np.ndarray:
    """One matrix step N(X) with coefficients (a_0, a_1, ..., a_d). In bf16
    mode the product operand is `operand` (the stored hi of the iterate) when
    given, else bf16(X)."""
    rd = rounding(mode)
    coeffs = [float(c) for c in coeffs]
    if mode != "exact" and len(coeffs) > 3:
        raise ValueError("the rounding contracts cover d <= 2")
    x = np.asarray(x, dtype=np.float64)
    tall = x.shape[0] >= x.shape[1]
    xo = rd(x) if operand is None else np.asarray(operand, dtype=np.float64)   # product operand
    g = xo.T @ xo if tall else xo @ xo.T
    d = len(coeffs) - 1
    if mode == "exact":
        b = np.zeros_like(g)
        gp = np.eye(g.shape[0])
        for i in range(1, d + 1):
            gp = gp @ g
            b = b + coeffs[i] * gp
    else:
        b = coeffs[1] * g
        if d == 2:
            gb = rd(g)
            b = b + coeffs[2] * (gb @ gb)
        b = rd(b)
    upd = xo @ b if tall else b @ xo
    return coeffs[0] * x + upd


def ns_filter(x0: np.ndarray, table, mode: str = "exact") -> np.ndarray:
    """N_L o ... o N_1 (X0) for a per-step coefficient table (eq:filter). In
    bf16 mode every step starts from the stored form (hi, e4m3 residual) of
    its input."""
    x = np.asarray(x0, dtype=np.float64)
    for row in table:
        if mode in ("exact", "f16"):
            x = ns_step(x, row, mode)
        else:
            hi, carried = store_state(x)
            x = ns_step(carried, row, mode, operand=hi)
    return x
