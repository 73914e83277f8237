"""IEEE single-precision fused multiply-add, computed exactly (test
infrastructure; only the tests, the smoke check and the benchmark's CPU
baseline use this package).

The score accumulator of the forward (Algorithm 1, the scaled product of the
quantized Q and K; Appendix C keeps it in fp32 before the FP16 softmax) adds
each 64-channel group's term with a fused multiply-add: a*b + c rounded once
to fp32.  numpy has no fused multiply-add, so it is built here from exact
float64 pieces:

  * p = a*b is exact in float64 (two 24-bit significands give at most 48
    bits);
  * s = fl64(p + c) and e = (p + c) - s, the exact rounding error of that
    addition (Knuth's TwoSum, exact for any two float64 values);
  * RN32(p + c) = RN32(s), except when s is exactly halfway between two fp32
    neighbours: then the sign of e says on which side of the tie p + c lies
    (e = 0 is a true tie, which the conversion already sends to even).
    If s is not such a midpoint, p + c lies within half a float64 ulp of s
    and cannot cross an fp32 midpoint, which is itself a float64 value.
"""
from __future__ import annotations

import numpy as np


def fma_f32(a, b, c):
    """RN32(a*b + c) for float32 a, b, c (broadcast); returns float32."""
    a = np.asarray(a, np.float32).astype(np.float64)
    b = np.asarray(b, np.float32).astype(np.float64)
    c = np.asarray(c, np.float32).astype(np.float64)
    p = a * b                                   # exact
    s = p + c
    bp = s - c                                  # TwoSum: s + e == p + c exactly
    bc = s - bp
    e = (p - bp) + (c - bc)
    r = s.astype(np.float32)
    up = np.nextafter(r, np.float32(np.inf))
    dn = np.nextafter(r, np.float32(-np.inf))
    r64 = r.astype(np.float64)
    mid_up = (r64 + up.astype(np.float64)) / 2  # exact in float64
    mid_dn = (r64 + dn.astype(np.float64)) / 2
    out = np.where((s == mid_up) & (e > 0), up, r)
    out = np.where((s == mid_dn) & (e < 0), dn, out)
    return out.astype(np.float32)
