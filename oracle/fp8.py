"""Decoding of OCP 8-bit floating point E4M3 ("e4m3fn") codes, in float64.

TEST INFRASTRUCTURE ONLY -- see the package docstring.

The fp8 variant of the cache stores each element as an E4M3 code plus one fp32
scale per (agent, layer, K or V, head); the stored value is code_value * scale.
This module gives code_value from the format's published definition (OCP
8-bit Floating Point Specification, E4M3): bit 7 sign, bits 6..3 exponent with
bias 7, bits 2..0 mantissa; exponent 0 encodes subnormals 2^-6 * m/8; the
single pattern S.1111.111 is NaN; there are no infinities; the largest finite
magnitude is 448.
"""

from __future__ import annotations

import numpy as np


def e4m3fn_decode(codes) -> np.ndarray:
    """Map uint8 E4M3 codes to their float64 values (NaN for the NaN codes)."""
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = c & 0x7
    normal = sign * np.ldexp(1.0 + m / 8.0, e - 7)
    sub = sign * np.ldexp(m / 8.0, -6)
    out = np.where(e == 0, sub, normal)
    return np.where((e == 15) & (m == 7), np.nan, out)


def e4m3fn_encode(x, scale) -> np.ndarray:
    """Quantise values to E4M3 codes against one scale: code = RNE(clamp(x / scale, -448, 448)).

    The quotient is taken in float32 (the precision the append kernel divides in), so both sides take the
    same integer decision from the same float32 value; the rounding to the E4M3 grid is exact here: every
    finite E4M3 value and every float32 value is a float64 value, so the distances below are exact.  Among
    the two nearest grid values a tie goes to the one with an even code (even mantissa), as round-to-
    nearest-even prescribes.  NaN inputs give the NaN code 0x7F (sign kept).
    """
    y = np.asarray(x, np.float32) / np.float32(scale)
    y = np.clip(y, np.float32(-448.0), np.float32(448.0)).astype(np.float64)
    grid_codes = np.arange(0x7F, dtype=np.uint8)  # 0x00 .. 0x7E: the non-negative finite values, increasing
    grid = e4m3fn_decode(grid_codes)
    a = np.abs(y).ravel()
    hi = np.searchsorted(grid, a, side="left").clip(0, len(grid) - 1)  # first grid value >= a
    lo = (hi - 1).clip(0, None)
    d_hi = grid[hi] - a
    d_lo = a - grid[lo]
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    idx = np.where(pick_hi, hi, lo)
    idx = np.where(a == grid[hi], hi, idx)
    code = grid_codes[idx].astype(np.uint8)
    neg = np.signbit(y.ravel())
    code = np.where(neg, code | 0x80, code)
    code = np.where(np.isnan(y.ravel()), np.where(neg, 0xFF, 0x7F), code)
    return code.astype(np.uint8).reshape(np.shape(x))
