"""Pins for the oracle's tiled forward (Algorithm 1, Theorem 1, Section 4.5).

  * with quantizers off and float64 state the online recurrence equals
    brute-force causal softmax attention (FlashAttention tiling, Background);
  * Theorem 1's closed forms for the consistent and mismatched normalizers,
    on the oracle's own quantized weights;
  * a constant V row is returned exactly under P-Reordering and scaled by
    (1 + eps) under the inconsistent normalizer;
  * one block: O equals the one-shot sum P^V^/sum P^ rebuilt from the dumped
    P^ codes;
  * causality, GQA mapping and the exactness of the group dots in fp32."""
import math

import numpy as np
import pytest

from oracle import attention, hif4, smooth
from paper_2607_04302_amd.workloads import small_case


def _brute(q, k, v, cu, hkv):
    """softmax(QK^T/sqrt(D) + causal mask) V per sequence/head in float64."""
    hq, d = q.shape[1], q.shape[2]
    out = np.zeros(q.shape)
    for b in range(len(cu) - 1):
        sl = slice(cu[b], cu[b + 1])
        L = cu[b + 1] - cu[b]
        mask = np.tril(np.ones((L, L), bool))
        for h in range(hq):
            qq = q[sl, h].astype(np.float64)
            kk = k[sl, h // (hq // hkv)].astype(np.float64)
            vv = v[sl, h // (hq // hkv)].astype(np.float64)
            s = qq @ kk.T / math.sqrt(d)
            s = np.where(mask, s, -np.inf)
            p = np.exp(s - s.max(1, keepdims=True))
            out[sl, h] = (p / p.sum(1, keepdims=True)) @ vv
    return out


@pytest.mark.parametrize("lens", [(1,), (63,), (64,), (65,), (200, 17, 130)])
def test_exact_mode_equals_softmax_attention(lens):
    q, k, v, cu = small_case(heads_q=4, heads_kv=2, head_dim=128, seqlens=lens, seed=11)
    ref = _brute(q, k, v, cu, 2)
    res = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, arith="exact")
    for (b, h), r in res.items():
        got = r["o"]
        want = ref[cu[b]:cu[b + 1], h]
        assert np.max(np.abs(got - want)) < 1e-12 * max(1.0, np.abs(want).max())


def test_fp16_contract_close_to_exact():
    q, k, v, cu = small_case(heads_q=2, heads_kv=1, seqlens=(300,), seed=2, outlier_channels=())
    ex = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, arith="exact")
    f16 = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, operands="fp16")
    for key in ex:
        assert np.max(np.abs(ex[key]["o"] - f16[key]["o"])) < 3e-3


def _thm1_terms(a, ahat, vrows):
    z = a.sum()
    w = a / z
    eps = ahat / a - 1.0
    ebar = (w * eps).sum()
    delta = eps - ebar
    ostar = w @ vrows
    e_t = (w * delta) @ (vrows - ostar)
    return ostar, ebar, delta, w, e_t


def test_theorem1_single_block():
    """Rows whose keys fit in one block: a_j = P16_j (offset m), a^_j = P^_j,
    v_j = V^ rows.  Check sum w delta = 0 and both closed forms."""
    q, k, v, cu = small_case(heads_q=1, heads_kv=1, seqlens=(64,), seed=4)
    res = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, want_p=True)[(0, 0)]
    res_mis = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, norm="inconsistent")[(0, 0)]
    _, vhat = attention.quantize_tokens(v[:, 0])
    qhat = attention.quantize_rows(q[:, 0])["xhat"].reshape(64, 128)
    khat = attention.quantize_rows(k[:, 0])["xhat"].reshape(64, 128)
    s2 = attention.scores_hif4(qhat, khat, 128)
    checked = 0
    for i in range(8, 64):
        keys = np.arange(i + 1)
        m = s2[i, keys].max()
        a = attention.exp2_fp16(attention.sub_fp16(s2[i, keys], m)).astype(np.float64)
        f = hif4.unpack(res["p_codes"][i, 0], res["p_meta"][i, 0])
        ahat = hif4.dequantize(f)[: i + 1]
        nz = a > 0
        a_, ah_, vr = a[nz], ahat[nz], vhat[keys][nz]
        # keys with a_j = 0 have a^_j = 0 and drop out of every sum
        assert np.all(ahat[~nz] == 0)
        ostar, ebar, delta, w, e_t = _thm1_terms(a_, ah_, vr)
        assert abs((w * delta).sum()) < 1e-13
        o_con = res["o"][i]
        o_mis = res_mis["o"][i]
        tol = 1e-12 * (1 + np.abs(ostar).max())
        assert np.max(np.abs((o_con - ostar) - e_t / (1 + ebar))) < tol
        assert np.max(np.abs((o_mis - ostar) - (e_t + ebar * ostar))) < tol
        assert np.max(np.abs(o_mis - (1 + ebar) * o_con)) < tol
        checked += 1
    assert checked > 40


def test_constant_v_exact_under_preorder():
    """Every key carries the same V row: P-Reordering returns V^ bit-exactly in
    fp16 across many blocks and rescales; the inconsistent normalizer returns
    (1 + eps) V^ with eps != 0 (Theorem 1 with e_t = 0)."""
    q, k, v, cu = small_case(heads_q=2, heads_kv=1, seqlens=(333,), seed=9)
    row = v[0, 0].copy()
    v[:] = row
    pre = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, norm="preorder", want_p=True)
    mis = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, norm="inconsistent")
    _, vhat = attention.quantize_tokens(v[:, 0])
    target = vhat[0].astype(np.float16)
    assert np.array_equal(vhat[0], target.astype(np.float64))
    n_diff = 0
    for key in pre:
        o16 = pre[key]["o16"]
        assert np.array_equal(o16, np.broadcast_to(target, o16.shape))
        ratio = pre[key]["l_con"] / pre[key]["l_mis"]          # 1 + eps per row
        om = mis[key]["o"]
        assert np.allclose(om, ratio[:, None] * vhat[0][None, :], rtol=1e-12, atol=1e-14)
        n_diff += np.sum(np.abs(ratio - 1) > 1e-6)
    assert n_diff > 100


def test_one_block_equals_one_shot_from_codes():
    q, k, v, cu = small_case(heads_q=1, heads_kv=1, seqlens=(50,), seed=21)
    r = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, want_p=True)[(0, 0)]
    _, vhat = attention.quantize_tokens(v[:, 0])
    phat = hif4.dequantize(hif4.unpack(r["p_codes"][:, 0], r["p_meta"][:, 0]))
    o = (phat @ vhat) / phat.sum(1, keepdims=True)
    assert np.max(np.abs(o - r["o"])) < 1e-12


def test_causality_and_gqa():
    q, k, v, cu = small_case(heads_q=4, heads_kv=2, seqlens=(150,), seed=5)
    base = attention.attention_fwd(q, k, v, None, cu_seqlens=cu)
    k2, v2 = k.copy(), v.copy()
    k2[100:] = np.float16(3.0)
    v2[100:] = np.float16(-2.0)
    alt = attention.attention_fwd(q, k2, v2, None, cu_seqlens=cu)
    for key in base:
        # rows before 100 never see the changed keys -- but V^ groups are 64
        # tokens wide, so rows in the block holding token 100 may change
        # through the shared V scale; rows < 64 are fully independent.
        assert np.array_equal(base[key]["o16"][:64], alt[key]["o16"][:64])
    # heads 0,1 share kv head 0; heads 2,3 share kv head 1
    q2 = q.copy()
    q2[:, 1] = q[:, 0]
    r = attention.attention_fwd(q2, k, v, None, cu_seqlens=cu, heads=[0, 1])
    assert np.array_equal(r[(0, 0)]["o16"], r[(0, 1)]["o16"])


def test_group_dots_exact_in_fp32():
    q, k, v, cu = small_case(heads_q=1, heads_kv=1, seqlens=(128,), seed=8)
    qhat = attention.quantize_rows(q[:, 0])["xhat"].reshape(128, 128)
    khat = attention.quantize_rows(k[:, 0])["xhat"].reshape(128, 128)
    for g in range(2):
        t = qhat[:, 64 * g:64 * g + 64] @ khat[:, 64 * g:64 * g + 64].T
        assert np.array_equal(t.astype(np.float32).astype(np.float64), t)


def test_smooth_scale_one_is_identity():
    q, k, v, cu = small_case(heads_q=2, heads_kv=1, seqlens=(100,), seed=6)
    ones = np.ones((1, 128), np.float32)
    a = attention.attention_fwd(q, k, v, ones, cu_seqlens=cu, want_p=True)
    b = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, want_p=True)
    for key in a:
        assert np.array_equal(a[key]["p_codes"], b[key]["p_codes"])
        assert np.array_equal(a[key]["o16"], b[key]["o16"])


def test_smoothing_preserves_qk_direction():
    """Q~ K~^T = Q K^T (Eq. 1, matrix form) up to the fp16 roundings of Q~ and
    K~; the wrong direction (K*s) would be off by the scale squared."""
    q, k, v, cu = small_case(heads_q=2, heads_kv=1, seqlens=(80,), seed=6)
    s = np.exp(np.random.default_rng(0).uniform(-1.5, 1.5, (1, 128))).astype(np.float32)
    qt, kt = smooth.apply(q, k, s, 1)
    for h in range(2):
        a = qt[:, h].astype(np.float64) @ kt[:, 0].astype(np.float64).T
        b = q[:, h].astype(np.float64) @ k[:, 0].astype(np.float64).T
        assert np.max(np.abs(a - b)) < 2e-2 * np.abs(b).max()


def test_score_rounding_goes_through_fp32():
    """S2 = fp16(fp32(S_acc * c)): the scaled score is rounded to fp32 first.
    Witness: S_acc = 1.386971354484558 (an fp32 value), D = 64.  The exact
    product S_acc * c lies above the fp16 midpoint M = 0.2501220703125 of
    0.25 and 0.250244140625 but rounds to M in fp32; rounding M to nearest
    even gives 0.25, while a single rounding of the exact product would give
    0.250244140625."""
    from fractions import Fraction
    s_acc = np.float32(1.386971354484558)
    c = attention.score_scale(64)
    mid = Fraction(0.25) + Fraction(1, 2 ** 13)
    assert Fraction(float(s_acc)) * Fraction(float(c)) > mid          # single rounding -> upper
    qhat = np.zeros((1, 64))
    khat = np.zeros((1, 64))
    qhat[0, 0] = float(s_acc)
    khat[0, 0] = 1.0
    s2 = attention.scores_hif4(qhat, khat, 64)
    assert s2.dtype == np.float16 and float(s2[0, 0]) == 0.25
