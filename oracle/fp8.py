"""OCP E4M3FN decoding from the bit formula (oracle).

The paper does not fix a KV precision; the fp8 workload stores keys and
values as OCP E4M3FN codes (1 sign bit, 4 exponent bits with bias 7, 3
mantissa bits; no infinities; S.1111.111 is NaN; largest finite value 448),
with one fp32 scale per physical block. Decoding, for code c:

    s = c >> 7, E = (c >> 3) & 15, M = c & 7
    E == 0      : (-1)^s * 2^(1-7) * (M / 8)        (subnormal)
    E == 15, M==7: NaN
    otherwise   : (-1)^s * 2^(E-7) * (1 + M / 8)
"""

from __future__ import annotations

import math

import numpy as np


def e4m3_value(code: int) -> float:
    """Value of one E4M3FN code, computed term by term."""
    s = (code >> 7) & 1
    e = (code >> 3) & 0xF
    m = code & 0x7
    sign = -1.0 if s else 1.0
    if e == 0xF and m == 0x7:
        return math.nan
    if e == 0:
        return sign * math.ldexp(m / 8.0, 1 - 7)
    return sign * math.ldexp(1.0 + m / 8.0, e - 7)


def e4m3_table() -> np.ndarray:
    """float32[256]: value of every code (exact: all fit in fp32)."""
    return np.array([e4m3_value(c) for c in range(256)], dtype=np.float32)
