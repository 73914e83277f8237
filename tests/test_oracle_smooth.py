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


def test_apply_rounding_contract():
    q = np.ones((1, 1, 64), np.float16)
    q[..., 1] = 3.0
    k = q.copy()
    s = np.full((1, 64), 3.0, np.float32)
    qt, kt = smooth.apply(q, k, s, 1)
    assert qt[0, 0, 1] == np.float16(9.0)
    assert kt[0, 0, 0] == np.float16(np.float32(1.0) / np.float32(3.0))
