"""Host emulations of arithmetic shortcuts the HIP kernels take, checked
exhaustively or on adversarial samples against the exact definitions.

* E6M2 base selection from the fp32 bits (smallest E6M2 value b with
  1.75 b >= A), for every positive finite fp16 A.
* The smoothed key RN16(k / s) from a reciprocal: RN16(RN32(k * RN32(1/s)))
  equals the correctly rounded quotient whenever the kernel's window test on
  the product's low mantissa bits does not send the element to the exact
  division.
* Element codes from the biased reciprocal step and one rounding onto the
  grid 2^-sh, for every fp16 magnitude, E6M2 base and shift in range.
"""
from fractions import Fraction

import numpy as np

from oracle import hif4


def _e6m2_ceil_bits(a32):
    bits = a32.view(np.uint32).astype(np.int64)
    mant = bits & 0x7FFFFF
    c = (mant > 0xC0000).astype(np.int64) + (mant > 0x280000) + (mant > 0x440000) + (mant > 0x600000)
    return 4 * (bits >> 23) - 387 + c


def test_e6m2_ceiling_from_bits_all_fp16():
    a = np.arange(1, 0x7C00, dtype=np.uint16).view(np.float16).astype(np.float32)
    code = _e6m2_ceil_bits(a)
    table = hif4.E6M2_TABLE.astype(np.float64)
    ref = np.searchsorted(1.75 * table, a.astype(np.float64), side="left")
    assert np.array_equal(code, ref)


def _rn16_exact(k, s):
    """Correctly rounded fp16 of the exact quotient k/s (k fp16, s fp32 > 0),
    by exact rational comparison against the two fp16 neighbours of the
    float64 quotient."""
    q = Fraction(float(k)) / Fraction(float(s))
    h = np.float16(float(q))
    lo, hi = sorted([h, np.nextafter(h, np.float16(np.inf) if Fraction(float(h)) < q else np.float16(-np.inf))],
                    key=float)
    dl, dh = q - Fraction(float(lo)), Fraction(float(hi)) - q
    if dl < dh:
        return lo
    if dh < dl:
        return hi
    return lo if (int(lo.view(np.uint16)) & 1) == 0 else hi


def _kernel_k_over_s(k, s):
    """(value, flagged): the reciprocal path and whether the window test sends
    the element to the exact division."""
    rs = np.float32(1.0) / np.float32(s)
    q = np.float32(np.float32(k) * rs)
    b = int(np.array(q, np.float32).view(np.uint32))
    near = ((b & 0x1FFF) - 0xFFD) & 0xFFFFFFFF < 7
    tiny = (b & 0x7F800000) < 0x38800000 and (b & 0x7FFFFFFF) != 0
    return np.float16(q), bool(near or tiny)


def test_reciprocal_quotient_matches_exact_rounding():
    rng = np.random.default_rng(11)
    k = (rng.standard_normal(20000) * rng.choice([0.01, 1.0, 30.0], 20000)).astype(np.float16)
    s = np.exp(rng.uniform(-3.0, 3.0, 20000)).astype(np.float32)
    # adversarial: quotients close to fp16 halfway points
    mids = rng.uniform(0.1, 100.0, 4000).astype(np.float16)
    ups = np.nextafter(mids, np.float16(np.inf))
    mid_val = (mids.astype(np.float64) + ups.astype(np.float64)) / 2
    s2 = np.exp(rng.uniform(-2.0, 2.0, 4000)).astype(np.float32)
    k2 = (mid_val * s2.astype(np.float64)).astype(np.float16)
    flagged = 0
    for kk, ss in list(zip(k, s)) + list(zip(k2, s2)):
        val, flag = _kernel_k_over_s(kk, ss)
        if flag:
            flagged += 1
            continue
        assert val == _rn16_exact(kk, ss) or (np.isinf(val) and np.isinf(_rn16_exact(kk, ss)))
    assert flagged < 0.05 * (len(k) + len(k2))


def _rcp_step_bits(code):
    """The kernels' reciprocal step R = (4/b)(1+2^-18), rounded, for E6M2
    base bytes `code`, built from the same fp32 constants and exponent add."""
    code = np.asarray(code, np.int64)
    m = code & 3
    lo = np.where(m & 1, 0x404CCD00, 0x40800020)
    hi = np.where(m & 1, 0x40124949, 0x402AAAD5)
    cb = np.where(m & 2, hi, lo)
    return ((cb + ((31 - (code >> 2)) << 23)) & 0xFFFFFFFF).astype(np.uint32).view(np.float32)


def test_element_rounding_all_fp16_all_bases():
    """Element codes as the kernels form them: the fused a*R + C_sh rounded
    once onto the grid 2^-sh (fp32 or fp16 destination alike) is
    u = round-half-even(a * R * 2^sh).  For every positive finite fp16 a, every
    E6M2 base b and every shift sh with a <= 1.75 b 2^-sh (the range the E2/E3
    decisions leave an element in), this must equal the definition
    u = round-half-away(a / step), step = b 2^-sh / 4, computed here in
    integers; exact ties must round up (that is what the 2^-18 bias in R is
    for)."""
    a_bits = np.arange(1, 0x7C00, dtype=np.uint16)
    a = a_bits.view(np.float16).astype(np.float64)
    a_int = np.round(a * 2.0 ** 24).astype(np.int64)            # a = a_int * 2^-24 exactly
    table = hif4.E6M2_TABLE.astype(np.float64)
    checked = ties = 0
    for code in range(256):
        b = table[code]
        e, m = code >> 2, code & 3
        R = float(_rcp_step_bits(code))
        for sh in range(3):
            sel = a <= 1.75 * b * 2.0 ** -sh
            if not sel.any():
                continue
            ai, av = a_int[sel], a[sel]
            u_kernel = np.rint(av * R * 2.0 ** sh)                # a*R exact in float64; rint = half-even
            # a / step = a_int * 2^(sh + 9 - e) * 4 / (4 + m); round half away in integers
            k = sh + 9 - e
            den = 4 + m
            if k >= 0:
                num = ai * (8 << k) + den
                u_ref = num // (2 * den)
                tie = (ai * (8 << k)) % (2 * den) == den
            else:
                sc = 1 << (-k)
                num = ai * 8 + den * sc
                u_ref = num // (2 * den * sc)
                tie = (ai * 8) % (2 * den * sc) == den * sc
            assert u_ref.max() <= 7
            bad = u_kernel.astype(np.int64) != u_ref
            assert not bad.any(), (code, sh, av[bad][:4], u_kernel[bad][:4], u_ref[bad][:4])
            checked += sel.sum()
            ties += tie.sum()
    assert checked > 10_000_000 and ties > 1000
