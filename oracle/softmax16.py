"""The FP16 softmax exponential (Appendix C, "FP16 operations": the running
maximum and the exponential exp(S - m) are kept in FP16; Algorithm 1 steps for
the running max, the rescale factor and P).

Scores are carried in base-2 units (log2(e) is folded into the score scale),
so exp(S - m) becomes 2^x.  The oracle's reading: E(x) = 2^x rounded once to
the nearest fp16 (ties to even), for any fp16 x; E(-inf) = 0.

float64 exp2 is accurate to about one float64 ulp, while every value 2^x with
x an fp16 number lies at least about 2^-25 (relative) from an fp16 rounding
midpoint (checked exhaustively against exact decimal arithmetic by the test
suite), so rounding the float64 result to fp16 is the exact E.
"""
from __future__ import annotations

import numpy as np


def exp2_fp16(x):
    """E(x) for fp16 x (any shape); returns fp16."""
    x = np.asarray(x, dtype=np.float16)
    with np.errstate(over="ignore", under="ignore"):
        return np.exp2(x.astype(np.float64)).astype(np.float16)


def sub_fp16(a, b):
    """fp16(a - b): the exact difference of two fp16 values rounded once."""
    with np.errstate(invalid="ignore", over="ignore"):
        return (np.asarray(a, np.float16).astype(np.float64)
                - np.asarray(b, np.float16).astype(np.float64)).astype(np.float16)
