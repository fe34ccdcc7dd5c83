"""bfloat16 round-to-nearest-even, written from the format's definition.

TEST INFRASTRUCTURE (see ``oracle/column.py``).

A bfloat16 number has an 8-bit significand (7 stored bits plus the implicit
one) and float32's exponent range. Rounding a float64 value keeps 8
significant bits: write x = m * 2^e with 0.5 <= |m| < 1 (frexp), scale the
significand to an integer grid of 2^8 steps, round half-to-even (np.rint),
and scale back. Below float32's smallest normal (2^-126) the grid is fixed at
2^-133, the bfloat16 subnormal spacing.
"""
from __future__ import annotations

import numpy as np


def round_bf16(x):
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    # normal numbers: 8 significant bits -> grid 2^(e-8)
    e = np.maximum(e, -125)  # subnormal range: fixed grid 2^-133
    q = np.rint(np.ldexp(x, 8 - e))
    out = np.ldexp(q, e - 8)
    # overflow to infinity above the largest finite bf16
    big = np.abs(out) > 3.3895313892515355e38
    if np.any(big):
        out = np.where(big, np.copysign(np.inf, x), out)
    return out
