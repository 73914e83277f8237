"""Pin for the oracle's FP16 softmax exponential E(x) = RN_fp16(2^x)
(paper: Appendix C, "FP16 operations"; Algorithm 1, rescale and P steps).

Checked exhaustively against exact decimal arithmetic: for every fp16 x in
[-26, 16] the oracle's value is the fp16 nearest to 2^x (ties to even), and no
2^x lies closer than 2^-30 (relative) to an fp16 rounding midpoint, which is
what lets the oracle round a float64 exp2."""
import decimal
from decimal import Decimal

import numpy as np

from oracle.softmax16 import exp2_fp16, sub_fp16

ALL = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).view(np.float16)


def _fp16_neighbors(v64):
    h = np.float16(v64)
    lo = h if float(h) <= v64 else np.nextafter(h, np.float16(0))
    hi = np.nextafter(lo, np.float16(np.inf))
    return lo, hi


def test_exp2_exhaustive_exact():
    ctx = decimal.Context(prec=50)
    ln2 = ctx.ln(Decimal(2))
    xs = ALL[np.isfinite(ALL) & (ALL >= -26) & (ALL <= 15.9)]
    got = exp2_fp16(xs)
    min_rel = 1.0
    for x, y in zip(xs, got):
        if float(x) == int(float(x)):
            ex = ctx.power(Decimal(2), int(float(x)))             # exact power
        else:
            ex = ctx.exp(ctx.multiply(Decimal(float(x)), ln2))    # 2^x, 50 digits
        lo, hi = _fp16_neighbors(float(ex))
        dlo, dhi = Decimal(float(lo)), Decimal(float(hi))
        mid = (dlo + dhi) / 2
        if ex < mid:
            want = lo
        elif ex > mid:
            want = hi
        else:  # exact tie cannot happen for non-integer x; integer x is exact
            want = lo if (lo.view(np.uint16) & 1) == 0 else hi
        assert y.view(np.uint16) == np.float16(want).view(np.uint16), (x, y, want)
        if ex != 0 and dhi != dlo and float(x) != int(float(x)):
            min_rel = min(min_rel, float(abs(ex - mid) / ex))
    assert min_rel > 2.0 ** -30, min_rel


def test_exp2_special_values():
    assert exp2_fp16(np.float16(-np.inf)) == 0
    assert exp2_fp16(np.float16(0)) == 1
    assert exp2_fp16(np.float16(-1)) == 0.5
    assert exp2_fp16(np.float16(-24)) == np.float16(2.0 ** -24)   # smallest subnormal
    assert exp2_fp16(np.float16(-26)) == 0                        # below half of it
    assert exp2_fp16(np.float16(-25)) == 0                        # tie 2^-25 -> even (0)


def test_sub_single_rounding():
    a = np.float16(1.0)
    b = np.float16(2.0 ** -12)          # exact difference needs 13 bits
    assert sub_fp16(a, b) == np.float16(1.0)   # rounds to nearest even
    assert sub_fp16(np.float16(-np.inf), np.float16(3)) == -np.inf
    assert sub_fp16(np.float16(5), np.float16(5)) == 0
