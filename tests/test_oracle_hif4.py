"""Pins for the oracle's HIF4 quantizer (paper: Background "HIF4"; Sec. 4.1).

Each test checks the float64 implementation against something other than
itself: exhaustive enumeration with exact rational arithmetic, invariants the
format must satisfy, and the 4.5 bits/value budget printed in the paper."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import hif4

ALL_FP16 = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).view(np.float16)
POS_FP16 = np.unique(ALL_FP16[np.isfinite(ALL_FP16) & (ALL_FP16 > 0)].astype(np.float64))


def _e6m2_fraction(byte):
    e, m = byte >> 2, byte & 3
    return Fraction(4 + m, 4) * (Fraction(2) ** (e - 31))


E6M2_FR = [_e6m2_fraction(b) for b in range(256)]


def test_bit_budget():
    # 64 four-bit elements + 32 bits of metadata = 4.5 bits per value
    assert hif4.BITS_PER_GROUP == 288
    assert hif4.BITS_PER_GROUP / 64 == 4.5
    f = hif4.quantize(np.linspace(-3, 3, 64))
    codes, meta = hif4.pack(f)
    assert codes.nbytes * 8 + meta.nbytes * 8 == 288


def test_e6m2_table_monotone_and_exact():
    assert np.all(np.diff(hif4.E6M2_TABLE) > 0)
    for b in (0, 1, 2, 3, 4, 124, 125, 127, 255):
        assert Fraction(hif4.E6M2_TABLE[b]) == E6M2_FR[b]


def test_base_scale_exhaustive():
    """Every positive fp16 group maximum A: the base is the smallest E6M2
    value b with 1.75*b >= A (linear scan in exact rationals)."""
    groups = np.zeros((POS_FP16.size, 64))
    groups[:, 0] = POS_FP16
    base = hif4.quantize(groups)["base"].astype(int)
    thr = [Fraction(7, 4) * v for v in E6M2_FR]
    for A, got in zip(POS_FP16, base):
        fa = Fraction(A)
        want = next(i for i in range(256) if thr[i] >= fa)
        assert got == want, (A, got, want)


@pytest.mark.parametrize("e", [31, 11, 40])
def test_element_code_exhaustive(e):
    """All fp16 magnitudes under a base of every mantissa at three exponents,
    in positions whose micro-exponent shift is 0, 1 or 2: the code equals the
    exact round-half-away-from-zero of |x|/step, and the shift equals the
    nested-halving rule, both evaluated in exact rationals."""
    for m in range(4):
        b = _e6m2_fraction(4 * e + m)
        A = Fraction(7, 4) * b
        if float(A) > 65504:
            continue
        cand = POS_FP16[POS_FP16 <= float(A)]
        n = cand.size
        g = np.zeros((3 * n, 64))
        g[:, 0] = float(A)                 # sets the base to exactly b
        g[0:n, 1] = cand                   # same 4-block as A: shift 0
        g[n:2 * n, 4] = cand               # 8-block 0, 4-block 1
        g[2 * n:, 8] = cand                # 8-block 1, 4-block 2
        f = hif4.quantize(g)
        assert np.all(f["base"] == 4 * e + m)
        pos = np.repeat([1, 4, 8], n)
        u = f["u"][np.arange(3 * n), pos]
        half = Fraction(7, 8) * b          # 0.875*b
        for i, a in enumerate(np.tile(cand, 3)):
            fa = Fraction(a)
            p = pos[i]
            if p == 1:
                sh = 0
            elif p == 4:
                sh = 1 if fa <= half else 0
            else:
                e2 = 1 if fa <= half else 0
                sh = e2 + (1 if fa <= half / (2 ** e2) else 0)
            step = b / (4 * 2 ** sh)
            q = fa / step
            want = int(q + Fraction(1, 2))   # floor(q + 1/2), q >= 0
            assert u[i] == want, (m, e, p, a, u[i], want)


def _random_groups(rng, n):
    x = rng.standard_normal((n, 64)).astype(np.float32)
    x[::3, rng.integers(0, 64)] *= 40          # outliers
    x[1::5, :32] *= 1e-3                       # wide intra-group range
    x[2::7] = 0.0                              # all-zero groups
    x[3::11, 5:40] = 0.0
    return x.astype(np.float16).astype(np.float64)


def test_invariants_random():
    rng = np.random.default_rng(3)
    x = _random_groups(rng, 4000)
    f = hif4.quantize(x)
    b = hif4.E6M2_TABLE[f["base"].astype(int)]
    shift = np.repeat(f["e2"], 8, -1).astype(int) + np.repeat(f["e3"], 4, -1)
    step = b[:, None] * 2.0 ** -shift / 4
    # rounding error at most half a step, and no clipping
    assert np.all(np.abs(x - f["xhat"]) <= step / 2)
    assert np.all(f["u"] <= 7)
    # sign symmetry
    fn = hif4.quantize(-x)
    assert np.array_equal(fn["xhat"], -f["xhat"])
    # scale equivariance by powers of two (stays inside fp16 and E6M2 ranges)
    for k in (-3, 1, 4):
        fk = hif4.quantize(x * 2.0 ** k)
        assert np.array_equal(fk["xhat"], f["xhat"] * 2.0 ** k)
    # pack/unpack/dequantize from the stored bits alone
    codes, meta = hif4.pack(f)
    g = hif4.unpack(codes, meta)
    for key in ("u", "sign", "base", "e2", "e3"):
        assert np.array_equal(g[key], f[key]), key
    assert np.array_equal(hif4.dequantize(g), f["xhat"])
    # +0 is canonical
    assert not np.any(f["sign"] & (f["u"] == 0))


def test_grid_groups_round_trip():
    """A group already on the HIF4 grid of a base b (values u*b/4, u in 0..7,
    with a 7 present so that b is the chosen base) is reproduced exactly: a
    sub-block small enough to get a halved scale holds only even codes of the
    coarse grid, which the finer grid also holds."""
    rng = np.random.default_rng(5)
    for e in (25, 31, 38):
        for m in range(4):
            b = hif4.E6M2_TABLE[4 * e + m]
            u = rng.integers(0, 8, (500, 64)).astype(np.float64)
            u[:, rng.integers(0, 64)] = 7
            sgn = rng.choice([-1.0, 1.0], (500, 64))
            x = sgn * u * b / 4
            f = hif4.quantize(x)
            assert np.all(f["base"] == 4 * e + m)
            assert np.array_equal(f["xhat"], x)


def test_halving_rule_matches_definition():
    """A sub-block max exactly at the half range (0.875*b) takes the halved
    scale; one fp16 ulp above keeps the full scale."""
    b = 1.0  # E6M2 byte 124
    g = np.zeros((2, 64))
    g[:, 0] = 1.75
    g[0, 8] = 0.875
    g[1, 8] = np.nextafter(np.float16(0.875), np.float16(1)).astype(np.float64)
    f = hif4.quantize(g)
    assert f["base"][0] == 124 and f["base"][1] == 124
    assert f["e2"][0, 1] and not f["e2"][1, 1]
    assert f["xhat"][0, 8] == 0.875
