"""Smooth-QK: calibration statistics, the applicability gate and the rescale.

Paper: Eq. 1 (Section 4.2) s_c = |Kmax_c|^alpha / |Qmax_c|^(1-alpha), applied
after RoPE as q*s and k/s; Section 4.3 and Section 5.1: the per-channel maxima
are RMS-aggregated over the calibration set; Appendix C (GQA): s is per
key-head channel and broadcast to the query heads of its group; Section 4.4 and
Table 1: the gate (Strong alpha=0.5 if rho_K >= 6 and T > 3, Mild alpha=0.25 if
rho_K >= 6 and 2 <= T <= 3, otherwise Bypass with s = 1).

Readings (the paper leaves these open):
  * per calibration sequence, Kmax[h,c] is the max over tokens of |K[:,h,c]|
    and Qmax[h,c] the max over tokens and over the query heads of group h;
    then the RMS over sequences; Eq. 1 in float64, rounded once to fp32;
  * a zero statistic, or a non-finite s, gives s = 1; Bypass gives s = 1;
  * gate statistics over every calibration element of the layer:
    rho_K = max|K| / P99(|K|) (linear-interpolation percentile),
    T = max|K| / max|Q|;
  * application: q~ = fp16(q * s) and k~ = fp16(k / s): the exact product or
    quotient of the fp16 activation and the fp32 scale, rounded once to fp16
    (round to nearest, ties to even).
"""
from __future__ import annotations

import numpy as np

BYPASS, MILD, STRONG = 0, 1, 2
ALPHA_OF_BRANCH = {BYPASS: 0.0, MILD: 0.25, STRONG: 0.5}


def gate(rho_k: float, t_kq: float) -> int:
    """Section 4.4 applicability gate; thresholds inclusive as printed."""
    if rho_k >= 6.0 and t_kq > 3.0:
        return STRONG
    if rho_k >= 6.0 and 2.0 <= t_kq <= 3.0:
        return MILD
    return BYPASS


def channel_stats(q_cal, k_cal, heads_kv):
    """Per-sequence max-abs statistics.  q_cal [n, S, Hq, D], k_cal [n, S, Hkv, D]
    (fp16).  Returns Qmax, Kmax float64 [n, Hkv, D]."""
    n, _, hq, d = q_cal.shape
    g = hq // heads_kv
    kmax = np.abs(k_cal.astype(np.float64)).max(axis=1)
    qa = np.abs(q_cal.astype(np.float64)).max(axis=1)          # [n, Hq, D]
    qmax = qa.reshape(n, heads_kv, g, d).max(axis=2)
    return qmax, kmax


def rms(x):
    """RMS over the calibration sequences (axis 0)."""
    return np.sqrt(np.mean(np.asarray(x, np.float64) ** 2, axis=0))


def gate_stats(q_cal, k_cal):
    ka = np.abs(k_cal.astype(np.float64)).ravel()
    kmax = ka.max()
    p99 = np.percentile(ka, 99.0)
    qmax = np.abs(q_cal.astype(np.float64)).max()
    rho = kmax / p99 if p99 > 0 else float("inf")
    t = kmax / qmax if qmax > 0 else float("inf")
    return float(rho), float(t)


def scales_from_stats(qbar, kbar, alpha):
    """Eq. 1 on aggregated statistics; float64 then one rounding to fp32."""
    with np.errstate(divide="ignore", invalid="ignore", over="ignore"):
        s = np.power(kbar, alpha) / np.power(qbar, 1.0 - alpha)
    bad = (kbar == 0) | (qbar == 0) | ~np.isfinite(s) | (s == 0)
    return np.where(bad, 1.0, s).astype(np.float32)


def calibrate(q_cal, k_cal, heads_kv, alpha):
    """alpha > 0: Eq. 1 with that alpha; alpha == 0: Bypass (s = 1);
    alpha < 0: the gate picks the branch.  Returns (s fp32 [Hkv, D], report)."""
    qmax, kmax = channel_stats(q_cal, k_cal, heads_kv)
    qbar, kbar = rms(qmax), rms(kmax)
    rho, t = gate_stats(q_cal, k_cal)
    if alpha < 0:
        branch = gate(rho, t)
        alpha_used = ALPHA_OF_BRANCH[branch]
    elif alpha == 0:
        branch, alpha_used = BYPASS, 0.0
    else:
        branch = STRONG if alpha >= 0.5 else MILD
        alpha_used = float(alpha)
    if alpha_used == 0.0:
        s = np.ones(kbar.shape, np.float32)
    else:
        s = scales_from_stats(qbar, kbar, alpha_used)
    return s, {"rho_k": rho, "t_kq": t, "branch": branch, "alpha_used": alpha_used,
               "qbar": qbar, "kbar": kbar}


def _round_quotient_fp16(k, s):
    """fp16 nearest to the exact quotient k/s (k fp16, s fp32), ties to even.
    The float64 quotient is within half a float64 ulp of the exact one, so it
    rounds to the same fp16 unless it lands exactly on an fp16 midpoint; there
    the exact sign of k - mid*s (mid*s is exact in float64) decides."""
    k64 = k.astype(np.float64)
    s64 = np.broadcast_to(s.astype(np.float64), k64.shape)
    with np.errstate(over="ignore", invalid="ignore", divide="ignore"):
        q64 = k64 / s64
        h = q64.astype(np.float16)
        hv = h.astype(np.float64)
        # neighbour on the far side of q64
        toward = np.where(q64 > hv, np.float16(np.inf), np.float16(-np.inf)).astype(np.float16)
        nb = np.nextafter(h, toward).astype(np.float64)
        mid = (hv + nb) / 2.0
        at_mid = np.isfinite(q64) & (q64 == mid) & (hv != nb)
        if np.any(at_mid):
            diff = k64 - mid * s64              # exact sign of (k/s - mid) * s
            exact_side = np.sign(diff) * np.sign(s64)
            want_nb = exact_side == np.sign(nb - mid)
            # an exact tie keeps the even neighbour, which astype already chose
            h = np.where(at_mid & want_nb & (diff != 0), nb.astype(np.float16), h)
    return h


def apply(q, k, s, heads_kv):
    """Smooth-QK on [..., H, D] fp16 tensors (q: Hq heads, k: Hkv heads)."""
    s = np.asarray(s, np.float32)
    hq = q.shape[-2]
    sq = np.repeat(s, hq // heads_kv, axis=0)
    # the product of an fp16 and an fp32 value is exact in float64
    qt = (q.astype(np.float64) * sq.astype(np.float64)).astype(np.float16)
    kt = _round_quotient_fp16(k, s)
    return qt, kt
