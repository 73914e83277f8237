"""Pins for Smooth-QK calibration and the gate (Eq. 1; Sections 4.2-4.4;
Tables 1 and 8)."""
import math
import os

import numpy as np
import pytest

from oracle import smooth

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _table1():
    rows = []
    for line in open(os.path.join(GOLD, "table1_gate.csv")):
        if line.startswith("#") or not line.strip():
            continue
        name, rho, t, act = line.strip().split(",")
        rows.append((name, float(rho), float(t), act))
    return rows


def test_gate_reproduces_table1():
    names = {"strong": smooth.STRONG, "mild": smooth.MILD, "bypass": smooth.BYPASS}
    rows = _table1()
    assert len(rows) == 5
    for name, rho, t, act in rows:
        assert smooth.gate(rho, t) == names[act], name


def test_gate_boundaries():
    assert smooth.gate(6.0, 3.0001) == smooth.STRONG
    assert smooth.gate(6.0, 3.0) == smooth.MILD
    assert smooth.gate(6.0, 2.0) == smooth.MILD
    assert smooth.gate(6.0, 1.999) == smooth.BYPASS
    assert smooth.gate(5.999, 14.0) == smooth.BYPASS
    assert smooth.ALPHA_OF_BRANCH[smooth.STRONG] == 0.5
    assert smooth.ALPHA_OF_BRANCH[smooth.MILD] == 0.25


def test_alpha_half_equalizes_magnitudes():
    """Section 4.2: with alpha = 0.5, |Kmax|/s = |Qmax|*s = sqrt(|Kmax||Qmax|)."""
    rng = np.random.default_rng(1)
    kbar = rng.uniform(0.5, 300, (4, 64))
    qbar = rng.uniform(0.5, 30, (4, 64))
    s = smooth.scales_from_stats(qbar, kbar, 0.5).astype(np.float64)
    gm = np.sqrt(kbar * qbar)
    assert np.allclose(kbar / s, gm, rtol=2e-7)
    assert np.allclose(qbar * s, gm, rtol=2e-7)
    s25 = smooth.scales_from_stats(qbar, kbar, 0.25).astype(np.float64)
    assert np.allclose(s25, kbar ** 0.25 / qbar ** 0.75, rtol=1e-7)


def test_table8_worked_example():
    """Qwen3-8B layer 0: the calibration-aggregate K maximum 220.8 under the
    scale 3.72 compresses to about 59 (=220.8/3.72); with alpha = 0.5 that
    scale implies |Qmax| = 220.8/3.72^2, and Eq. 1 must return 3.72 for it."""
    vals = {}
    for line in open(os.path.join(GOLD, "table8_smooth_layer0.txt")):
        if line.startswith("#") or not line.strip():
            continue
        kk, vv = line.split()
        vals[kk] = float(vv)
    kbar = np.array([vals["kmax"]])
    qbar = kbar / vals["s"] ** 2
    s = smooth.scales_from_stats(qbar, kbar, 0.5)
    assert abs(float(s[0]) - vals["s"]) < 1e-5
    compressed = np.float32(np.float16(vals["kmax"])) / s[0]
    assert round(float(compressed)) == vals["compressed_approx"]
    assert abs(vals["kmax"] / vals["p99"] - vals["rho_k"]) < 0.05


def test_rms_aggregation_and_group_max():
    """Per-sequence maxima, query maxima over the group's heads, then the RMS
    over sequences (Sections 4.3 and 5.1; Appendix C for GQA)."""
    n, S, hq, hkv, d = 3, 10, 4, 2, 64
    q = np.zeros((n, S, hq, d), np.float16)
    k = np.zeros((n, S, hkv, d), np.float16)
    kmax = np.array([2.0, 4.0, 8.0])
    for i in range(n):
        k[i, 3, 1, 7] = -kmax[i]
        q[i, 5, 3, 7] = i + 1.0          # head 3 belongs to kv head 1
    qm, km = smooth.channel_stats(q, k, hkv)
    assert km[:, 1, 7].tolist() == kmax.tolist()
    assert qm[:, 1, 7].tolist() == [1.0, 2.0, 3.0]
    assert qm[:, 0, 7].tolist() == [0.0, 0.0, 0.0]
    assert math.isclose(smooth.rms(km)[1, 7], math.sqrt((4 + 16 + 64) / 3))
    s, rep = smooth.calibrate(q, k, hkv, 0.5)
    assert s[1, 7] == np.float32(math.sqrt(math.sqrt(28.0) / math.sqrt(14.0 / 3)))
    assert s[0, 0] == 1.0                # zero statistics -> s = 1


def test_bypass_and_gate_pick():
    rng = np.random.default_rng(2)
    q = rng.standard_normal((2, 64, 2, 64)).astype(np.float16)
    k = rng.standard_normal((2, 64, 1, 64)).astype(np.float16)
    s, rep = smooth.calibrate(q, k, 1, 0.0)
    assert np.all(s == 1) and rep["branch"] == smooth.BYPASS
    s, rep = smooth.calibrate(q, k, 1, -1.0)   # gaussian K: rho < 6 -> bypass
    assert rep["branch"] == smooth.BYPASS and np.all(s == 1)
    k2 = k.copy()
    k2[0, 0, 0, 5] = 200.0                      # one concentrated outlier
    s, rep = smooth.calibrate(q, k2, 1, -1.0)
    assert rep["rho_k"] >= 6 and rep["t_kq"] > 3 and rep["branch"] == smooth.STRONG
    assert s[0, 5] > 1


def _rn16_exact(fr):
    """fp16 nearest to a Fraction (ties to even), by exact comparison."""
    from fractions import Fraction
    h = np.float16(float(fr))
    cands = [np.nextafter(h, np.float16(-np.inf)), h, np.nextafter(h, np.float16(np.inf))]
    best = min(cands, key=lambda c: (abs(Fraction(float(c)) - fr), int(c.view(np.uint16)) & 1))
    return best


def test_apply_single_rounding_exhaustive_sample():
    """q~ = fp16(q*s) and k~ = fp16(k/s) are the exact product and quotient
    rounded once; checked with exact rationals on random operands and on
    operands built so that an fp32 intermediate would sit on an fp16 midpoint
    (where rounding twice would differ)."""
    from fractions import Fraction
    rng = np.random.default_rng(11)
    q = rng.standard_normal((1, 400, 1, 64)).astype(np.float16)
    s = np.exp(rng.uniform(-3, 3, (1, 64))).astype(np.float32)
    qt, kt = smooth.apply(q, q, s, 1)
    for i in range(0, 400, 7):
        for c in range(0, 64, 5):
            fq, fs = Fraction(float(q[0, i, 0, c])), Fraction(float(s[0, c]))
            assert qt[0, i, 0, c] == _rn16_exact(fq * fs)
            assert kt[0, i, 0, c] == _rn16_exact(fq / fs)
    # k/s whose fp32 rounding lands exactly on an fp16 midpoint: s is the fp32
    # nearest to k/M for a midpoint M, so the fp32 quotient is M itself while
    # the exact quotient is not
    found = differ = 0
    for kv in np.arange(1.0, 2.0, 2.0 ** -6).astype(np.float16):
        base = np.float16(float(kv) / 1.3)
        mid = (float(base) + float(np.nextafter(base, np.float16(2)))) / 2
        sv = np.float32(float(kv) / mid)
        q32 = np.float32(kv) / sv
        if float(q32) != mid or Fraction(float(kv)) / Fraction(float(sv)) == Fraction(mid):
            continue
        found += 1
        one = np.full((1, 1, 1, 64), kv, np.float16)
        got = smooth.apply(one, one, np.full((1, 64), sv, np.float32), 1)[1]
        want = _rn16_exact(Fraction(float(kv)) / Fraction(float(sv)))
        assert got[0, 0, 0, 0] == want
        differ += want != np.float16(q32)   # cases where rounding twice is wrong
    assert found > 0 and differ > 0
