"""Rounding used by the oracle's bf16 and fp16 contract modes.

The paper trains in bfloat16 (Sec. 3 setup) but does not fix where values are
rounded. The library's contract (and this mode) rounds to bfloat16 exactly at
the operands of the bf16 matrix products and at the stored iterate; all other
arithmetic here is float64.
"""
from __future__ import annotations

import numpy as np


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 (8 significant bits, ties
    to even), returned as float64. Exponent range as float32; no overflow
    handling is needed for the values this package produces."""
    x = np.asarray(x, dtype=np.float64)
    mant, expo = np.frexp(x)                 # x = mant * 2**expo, |mant| in [0.5, 1)
    expo = np.maximum(expo, -125)            # bf16 subnormal spacing 2**-133
    q = np.ldexp(x, 8 - expo)                # |q| < 2**8 for normal values
    return np.ldexp(np.rint(q), expo - 8)    # np.rint rounds half to even


E4M3_MAX = 448.0


def round_e4m3(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest OCP float8 e4m3 ("fn") value (3
    fraction bits, exponent bias 7, subnormal spacing 2**-9, largest finite
    448), ties to even, returned as float64. Inputs must lie in [-448, 448]
    (callers clamp first; the format has no infinities)."""
    x = np.asarray(x, dtype=np.float64)
    if np.any(np.abs(x) > E4M3_MAX):
        raise ValueError("round_e4m3 takes values in [-448, 448]")
    mant, expo = np.frexp(x)                 # x = mant * 2**expo, |mant| in [0.5, 1)
    expo = np.maximum(expo, -5)              # normal range starts at 2**-6
    q = np.ldexp(x, 4 - expo)                # |q| < 2**4
    return np.ldexp(np.rint(q), expo - 4)    # np.rint rounds half to even


F16_MAX = 65504.0


def round_f16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest IEEE binary16 value (10 fraction
    bits, subnormal spacing 2**-24), ties to even, returned as float64. Inputs
    must lie within the format's finite range (the filter's operands do)."""
    x = np.asarray(x, dtype=np.float64)
    if np.any(np.abs(x) > F16_MAX):
        raise ValueError("round_f16 takes values in [-65504, 65504]")
    mant, expo = np.frexp(x)                 # x = mant * 2**expo, |mant| in [0.5, 1)
    expo = np.maximum(expo, -13)             # normal range starts at 2**-14
    q = np.ldexp(x, 11 - expo)               # |q| < 2**11
    return np.ldexp(np.rint(q), expo - 11)   # np.rint rounds half to even


def identity(x: np.ndarray) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


def rounding(mode: str):
    if mode == "exact":
        return identity
    if mode == "bf16":
        return round_bf16
    if mode == "f16":
        return round_f16
    raise ValueError(f"unknown precision mode {mode!r}")
