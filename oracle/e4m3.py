"""OCP 8-bit floating point E4M3FN decode (test infrastructure only).

The paper deploys with FP8 post-training quantisation (Section "Experiments",
Deployment paragraph; Table 1, "LiteVLM in FP8" row) without naming the format;
the reading taken here is OCP E4M3FN, the format of the gfx950 matrix cores:
1 sign bit, 4 exponent bits with bias 7, 3 mantissa bits, subnormals when the
exponent field is 0, no infinities, NaN only for the codes S.1111.111, largest
finite magnitude 448.
"""
from __future__ import annotations

import math

import numpy as np


def decode_byte(code: int) -> float:
    """Value of one E4M3FN byte, from the definition above."""
    sign = -1.0 if (code >> 7) & 1 else 1.0
    exp = (code >> 3) & 0xF
    man = code & 0x7
    if exp == 0xF and man == 0x7:
        return math.nan
    if exp == 0:
        return sign * math.ldexp(man / 8.0, 1 - 7)
    return sign * math.ldexp(1.0 + man / 8.0, exp - 7)


DECODE_TABLE = np.array([decode_byte(c) for c in range(256)], dtype=np.float64)


def decode(bytes_: np.ndarray, scale: float = 1.0) -> np.ndarray:
    """Exact float64 values of E4M3FN bytes times a per-tensor scale."""
    return DECODE_TABLE[np.asarray(bytes_, dtype=np.uint8)] * np.float64(scale)
