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
