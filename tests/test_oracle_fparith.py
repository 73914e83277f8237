"""Pins for the oracle's fp32 fused multiply-add (the score accumulator's
per-group step): every result equals the exact rational a*b + c rounded once
to fp32 (nearest, ties to even), including values constructed to sit exactly
on, just above and just below fp32 rounding midpoints, where a separate
product and sum (two roundings) or a float64 sum rounded to fp32 (double
rounding) would differ."""
from fractions import Fraction

import numpy as np

from oracle.fparith import fma_f32
from tests.test_oracle_attention import _rn32


def _check(a, b, c):
    got = fma_f32(a, b, c)
    for x, y, z, r in zip(a.ravel(), b.ravel(), c.ravel(), got.ravel()):
        want = _rn32(Fraction(float(x)) * Fraction(float(y)) + Fraction(float(z)))
        assert Fraction(float(r)) == want, (x, y, z, r, float(want))


def test_random_operands():
    rng = np.random.default_rng(0)
    n = 3000
    a = (rng.standard_normal(n) * np.exp2(rng.integers(-20, 20, n))).astype(np.float32)
    b = (rng.standard_normal(n) * np.exp2(rng.integers(-20, 20, n))).astype(np.float32)
    c = (rng.standard_normal(n) * np.exp2(rng.integers(-40, 40, n))).astype(np.float32)
    _check(a, b, c)


def test_midpoints_and_their_neighbours():
    """c = -fp32(a*b) + (half an ulp of the result) +- tiny: p + c lands on,
    above or below an fp32 midpoint, and the float64 sum alone is not enough
    to decide."""
    rng = np.random.default_rng(1)
    a_l, b_l, c_l = [], [], []
    for _ in range(600):
        a = np.float32(1.0 + rng.integers(1, 2 ** 23) * 2.0 ** -23)
        b = np.float32(1.0 + rng.integers(1, 2 ** 23) * 2.0 ** -23)
        r = np.float32(np.float32(a) * np.float32(b))
        # p = a*b exactly; choose c = fp32 value near M - p, M a midpoint of r
        p = Fraction(float(a)) * Fraction(float(b))
        ulp = Fraction(float(np.nextafter(r, np.float32(np.inf)))) - Fraction(float(r))
        for off in (ulp / 2, -ulp / 2):
            target = Fraction(float(r)) + off + 8 * ulp - p     # distance to a midpoint of r + 8 ulp
            for shift in (0, 1, -1):
                cz = np.float32(float(target))
                cz = np.float32(np.nextafter(cz, np.float32(np.inf)) if shift > 0 else
                                (np.nextafter(cz, np.float32(-np.inf)) if shift < 0 else cz))
                a_l.append(a); b_l.append(b); c_l.append(cz)
    _check(np.array(a_l, np.float32), np.array(b_l, np.float32), np.array(c_l, np.float32))


def test_exact_ties_go_to_even():
    # 1 + 2^-24 is the midpoint of 1 and 1 + 2^-23: ties to even gives 1
    a = np.array([1.0 + 2.0 ** -12], np.float32)
    b = np.array([1.0 + 2.0 ** -12], np.float32)      # a*b = 1 + 2^-11 + 2^-24
    c = np.array([-2.0 ** -11], np.float32)
    assert float(fma_f32(a, b, c)[0]) == 1.0
    # 1 + 3*2^-24 is the midpoint of 1 + 2^-23 and 1 + 2^-22: even is 1 + 2^-22
    c2 = np.array([-2.0 ** -11 + 2.0 ** -23], np.float32)
    assert float(fma_f32(a, b, c2)[0]) == 1.0 + 2.0 ** -22
