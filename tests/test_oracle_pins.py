"""Pins for oracle functions that the other pin files leave open.

  * LSE (the log of the softmax partition, natural log): with quantizers off
    it equals a float64 brute-force log-sum-exp of QK^T/sqrt(D) over the
    causal keys; on the quantized path it equals m*ln2 + ln(l) with l rebuilt
    from the dumped P^ codes and the fp16 rescale factors of the running
    maximum (Algorithm 1's recurrence unrolled), for both normalizers; for
    the first query row it has the closed form S2*ln2 + ln(15/16);
  * HIF4 of V along tokens (groups of 64 consecutive tokens of one channel,
    aligned to each sequence's first token, a partial last group zero
    padded): on a constructed V whose groups each hold one planted outlier,
    every code, base and micro-exponent is known in closed form; a grouping
    along channels, a group aligned to the packed token index or a missing
    pad changes them;
  * the gate's P99 uses linear interpolation between order statistics
    (hand-computed value); nearest-rank would give another rho_K;
  * the canonical packed layout against bytes written from the layout's
    definition (32 code bytes, element 2i in the low nibble of byte i,
    nibble = sign<<3 | u; then base | E2 << 8 | E3 << 16, little endian);
  * fp16(a - b) is one rounding of the exact difference, including pairs
    whose difference rounded to fp32 first would land on an fp16 midpoint."""
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import attention, hif4, smooth
from oracle.softmax16 import exp2_fp16, sub_fp16
from paper_2607_04302_amd.workloads import small_case

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _brute_lse(q, k, cu, hkv):
    hq, d = q.shape[1], q.shape[2]
    out = {}
    for b in range(len(cu) - 1):
        sl = slice(cu[b], cu[b + 1])
        L = cu[b + 1] - cu[b]
        for h in range(hq):
            s = q[sl, h].astype(np.float64) @ k[sl, h // (hq // hkv)].astype(np.float64).T / math.sqrt(d)
            s = np.where(np.tril(np.ones((L, L), bool)), s, -np.inf)
            mx = s.max(1)
            out[(b, h)] = mx + np.log(np.exp(s - mx[:, None]).sum(1))
    return out


@pytest.mark.parametrize("lens", [(1,), (63,), (64,), (65,), (200, 17, 130)])
def test_lse_exact_mode_equals_logsumexp(lens):
    q, k, v, cu = small_case(heads_q=4, heads_kv=2, head_dim=128, seqlens=lens, seed=31)
    ref = _brute_lse(q, k, cu, 2)
    res = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, arith="exact")
    for key, r in res.items():
        assert r["lse"].dtype == np.float32
        assert np.max(np.abs(r["lse"] - ref[key])) <= 2e-6 * max(1.0, np.abs(ref[key]).max())


@pytest.mark.parametrize("norm", ["preorder", "inconsistent"])
def test_lse_rebuilt_from_dumped_codes(norm):
    """l = sum_J R_J sum_k a_Jk, with R_J the product of the fp16 rescale
    factors E(fp16(m_{J'-1} - m_J')) of the blocks after J, a = P^ (from the
    dumped codes) or P16 (inconsistent), and m_J the running maximum after
    block J."""
    q, k, v, cu = small_case(heads_q=2, heads_kv=1, head_dim=128, seqlens=(300,), seed=32)
    s = np.exp(np.random.default_rng(32).uniform(-1, 1, (1, 128))).astype(np.float32)
    res = attention.attention_fwd(q, k, v, s, cu_seqlens=cu, norm=norm, want_p=True)
    qt, kt = smooth.apply(q, k, s, 1)
    for h in range(2):
        r = res[(0, h)]
        qf = attention.quantize_rows(qt[:, h])
        khat = attention.quantize_rows(kt[:, 0])["xhat"].reshape(300, 128)
        s2 = attention.scores_hif4(attention.unit_operands(qf).reshape(300, 128), qf["scale"], khat, 128)
        for i in (0, 5, 63, 64, 130, 299):
            nb = i // 64 + 1
            row = np.where(np.arange(300) <= i, s2[i], np.float16(-np.inf)).astype(np.float16)
            bm = [row[64 * J:64 * J + 64].max() for J in range(nb)]
            m = [np.float16(-np.inf)]
            for J in range(nb):
                m.append(max(m[-1], bm[J]))
            l = 0.0
            for J in range(nb):
                rj = float(exp2_fp16(sub_fp16(m[J], m[J + 1]))) if J > 0 else 0.0
                blk = row[64 * J:64 * J + 64]
                if norm == "preorder":
                    a = hif4.dequantize(hif4.unpack(r["p_codes"][i, J], r["p_meta"][i, J]))
                else:
                    a = exp2_fp16(sub_fp16(blk, m[J + 1])).astype(np.float64)
                l = l * rj + a.sum()
            want = float(m[-1]) * math.log(2.0) + math.log(l)
            assert abs(float(r["lse"][i]) - want) <= 1e-6 * max(1.0, abs(want)), (h, i)


def test_lse_first_row_closed_form():
    """Row 0 sees one key: P16 = 2^0 = 1, whose HIF4 group has base 0.625 (the
    smallest E6M2 value with 1.75 b >= 1) and code round(1 / 0.15625) = 6, so
    P^ = 0.9375 and LSE = S2*ln 2 + ln(15/16)."""
    q, k, v, cu = small_case(heads_q=1, heads_kv=1, head_dim=64, seqlens=(10,), seed=33)
    r = attention.attention_fwd(q, k, v, None, cu_seqlens=cu)[(0, 0)]
    qf = attention.quantize_rows(q[:, 0])
    khat = attention.quantize_rows(k[:, 0])["xhat"].reshape(10, 64)
    s2 = attention.scores_hif4(attention.unit_operands(qf).reshape(10, 64), qf["scale"], khat, 64)
    want = float(s2[0, 0]) * math.log(2.0) + math.log(15.0 / 16.0)
    assert abs(float(r["lse"][0]) - want) <= 1e-6 * max(1.0, abs(want))


def _planted_v(lens, hkv, d, seed):
    """V [T, Hkv, D] (THD) that is zero except one outlier per (sequence,
    token group, head, channel): value +-1.75 * 2^e at a random position of
    the group's valid tokens.  Returns V and the list of plants."""
    rng = np.random.default_rng(seed)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    v = np.zeros((int(cu[-1]), hkv, d), np.float16)
    plants = []
    for b, L in enumerate(lens):
        for g in range(-(-L // 64)):
            n_valid = min(64, L - 64 * g)
            for h in range(hkv):
                for c in range(d):
                    pos = int(rng.integers(0, n_valid))
                    e = int(rng.integers(-6, 6))
                    neg = bool(rng.integers(0, 2))
                    v[cu[b] + 64 * g + pos, h, c] = (-1.75 if neg else 1.75) * 2.0 ** e
                    plants.append((b, g, h, c, pos, e, neg))
    return v, cu, plants


def _expected_group(pos, e, neg):
    """Closed form for a group that is zero except +-1.75*2^e at `pos`: base
    2^e (byte (e+31)<<2), code 7 there; every 8-block without the outlier
    and every 4-block without it have their bit set (max 0 fits)."""
    codes = np.zeros(32, np.uint8)
    nib = (8 if neg else 0) | 7
    codes[pos // 2] = nib << (4 * (pos % 2))
    e2 = 0xFF & ~(1 << (pos // 8))
    e3 = 0xFFFF & ~(1 << (pos // 4))
    meta = ((e + 31) << 2) | (e2 << 8) | (e3 << 16)
    return codes, np.uint32(meta)


def test_v_groups_run_along_tokens_from_each_sequence_start():
    lens = (130, 64, 1, 77)          # ragged tails, an exact group, one token; starts at 0, 130, 194, 195
    hkv, d = 2, 64
    v, cu, plants = _planted_v(lens, hkv, d, seed=34)
    codes, metas = attention.quantize_v(v, cu)
    n_groups = sum(-(-L // 64) for L in lens)
    assert codes.shape == (n_groups, hkv, d, 32) and metas.shape == (n_groups, hkv, d)
    gidx = {}
    for b, L in enumerate(lens):
        for g in range(-(-L // 64)):
            gidx[(b, g)] = len(gidx)
    for (b, g, h, c, pos, e, neg) in plants:
        want_c, want_m = _expected_group(pos, e, neg)
        G = gidx[(b, g)]
        assert np.array_equal(codes[G, h, c], want_c), (b, g, h, c)
        assert metas[G, h, c] == want_m, (b, g, h, c)
    # V^ is V itself here (every value on the grid), zero padded per sequence
    for b, L in enumerate(lens):
        f, vhat = attention.quantize_tokens(v[cu[b]:cu[b + 1], 0])
        lp = -(-L // 64) * 64
        assert vhat.shape == (lp, d)
        assert np.array_equal(vhat[:L], v[cu[b]:cu[b + 1], 0].astype(np.float64))
        assert np.all(vhat[L:] == 0)


def test_gate_p99_interpolates_linearly():
    """|K| = 1, 2, ..., 100: the 99th percentile by linear interpolation is
    x[98] + 0.01 (x[99] - x[98]) = 99.01 (nearest rank would give 99 or 100),
    so rho_K = 100 / 99.01; T = max|K| / max|Q| = 100 / 4."""
    k = np.arange(1, 101, dtype=np.float16).reshape(1, 100, 1, 1)
    k[0, ::2] *= -1
    q = np.full((1, 100, 1, 1), 4.0, np.float16)
    q[0, 7] = -4.0
    rho, t = smooth.gate_stats(q, k)
    assert rho == pytest.approx(100.0 / 99.01, rel=1e-14)
    assert t == 25.0


def _golden_bytes(name):
    with open(os.path.join(GOLD, name)) as f:
        return bytes.fromhex("".join(l.split("#")[0].strip() for l in f))


def test_pack_matches_the_layout_bytes():
    u = np.array([k % 8 for k in range(64)], np.uint8)
    sign = np.array([16 <= k < 32 and k % 8 != 0 for k in range(64)])
    e2 = np.array([(0xA5 >> j) & 1 for j in range(8)], bool)
    e3 = np.array([(0x1234 >> j) & 1 for j in range(16)], bool)
    fields = {"u": u[None], "sign": sign[None], "base": np.array([0x7C], np.uint8),
              "e2": e2[None], "e3": e3[None]}
    codes, meta = hif4.pack(fields)
    got = codes[0].tobytes() + meta.astype("<u4")[0].tobytes()
    assert got == _golden_bytes("hif4_pack_layout.hex")
    back = hif4.unpack(codes, meta)
    for key in ("u", "sign", "base", "e2", "e3"):
        assert np.array_equal(back[key], fields[key]), key


def _rn16(x):
    if x == 0:
        return Fraction(0)
    a = abs(x)
    e = max(a.numerator.bit_length() - a.denominator.bit_length() - (1 if Fraction(2) ** (a.numerator.bit_length() - a.denominator.bit_length()) > a else 0), -14)
    ulp = Fraction(2) ** (e - 10)
    q, r = divmod(a, ulp)
    if r * 2 > ulp or (r * 2 == ulp and q % 2 == 1):
        q += 1
    return (1 if x > 0 else -1) * q * ulp


def test_sub_fp16_rounds_the_exact_difference_once():
    """20000 random finite fp16 pairs over every exponent combination against
    the exact rational difference rounded once to fp16 (ties to even);
    plus the special cases.  (An fp32 subtraction followed by a conversion
    to fp16 gives the same value: 24 >= 2*11 + 2 significant bits make that
    double rounding innocuous, so the GPU's fp16 subtraction needs no
    special care either; the sweep checks it.)"""
    rng = np.random.default_rng(35)
    bits = rng.integers(0, 0x7C00, size=(20000, 2)).astype(np.uint16)
    a = bits[:, 0].view(np.float16)
    b = bits[:, 1].view(np.float16)
    b = np.where(rng.integers(0, 2, 20000) == 1, b, -b).astype(np.float16)
    got = sub_fp16(a, b)
    with np.errstate(over="ignore"):
        via32 = (a.astype(np.float32) - b.astype(np.float32)).astype(np.float16)
    n = 0
    for x, y, g, t in zip(a, b, got, via32):
        exact = Fraction(float(x)) - Fraction(float(y))
        want = _rn16(exact)
        if abs(want) > 65504:
            assert np.isinf(g) and np.sign(g) == np.sign(float(exact))
            continue
        assert Fraction(float(g)) == want, (x, y)
        assert Fraction(float(t)) == want, (x, y)
        n += 1
    assert n > 19000
    assert sub_fp16(np.float16(-np.inf), np.float16(3)) == -np.inf
    assert sub_fp16(np.float16(5), np.float16(5)) == 0 and not np.signbit(sub_fp16(np.float16(5), np.float16(5)))
    assert float(sub_fp16(np.float16(2.0 ** -14), np.float16(2.0 ** -24))) == 2.0 ** -14 - 2.0 ** -24   # subnormal
    assert float(sub_fp16(np.float16(1.0), np.float16(2.0 ** -12))) == 1.0          # tie to even
    assert float(sub_fp16(np.float16(1.0), np.float16(-2.0 ** -11))) == 1.0         # tie to even
    assert float(sub_fp16(np.float16(1.0), np.float16(-3 * 2.0 ** -11))) == 1.0 + 2.0 ** -9
