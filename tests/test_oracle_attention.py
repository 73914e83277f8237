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
    qf = attention.quantize_rows(q[:, 0])
    khat = attention.quantize_rows(k[:, 0])["xhat"].reshape(64, 128)
    s2 = attention.scores_hif4(attention.unit_operands(qf).reshape(64, 128), qf["scale"], khat, 128)
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


def _rn(x, bits, emin):
    """x (a Fraction) rounded to the nearest binary float with `bits`
    significant bits and minimum normal exponent emin (ties to even)."""
    from fractions import Fraction
    if x == 0:
        return Fraction(0)
    sgn = -1 if x < 0 else 1
    a = abs(x)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    e = max(e, emin)
    ulp = Fraction(2) ** (e - bits + 1)
    q, r = divmod(a, ulp)
    if r * 2 > ulp or (r * 2 == ulp and q % 2 == 1):
        q += 1
    return sgn * q * ulp


def _rn32(x):
    return _rn(x, 24, -126)


def _rn16(x):
    return _rn(x, 11, -14)


def _one_term(d, head_dim):
    """q_op/q_base/khat arrays whose group dots are d (one term per group)."""
    g = len(d)
    q_op = np.zeros((1, head_dim))
    khat = np.zeros((1, head_dim))
    for i, dv in enumerate(d):
        q_op[0, 64 * i] = 1.0
        khat[0, 64 * i] = dv
    return q_op, khat


def test_score_rounds_to_fp32_then_fp16():
    """S2 = fp16(fp32(S_acc * c)): the scaled score is an fp32 value before the
    conversion to fp16.  Witness (D = 64, one group term d with base 4, so
    S_acc = d): d = 1.386971354484558 (an fp32 value); the exact product d*c
    lies above the fp16 midpoint M = 0.2501220703125 of 0.25 and
    0.250244140625 but rounds to M in fp32; M then rounds to the even 0.25,
    while a single rounding of the exact product would give 0.250244140625."""
    from fractions import Fraction
    d = float(np.float32(1.386971354484558))
    c = attention.score_scale(64)
    exact = Fraction(d) * Fraction(float(c))
    assert _rn16(exact) == Fraction(0.250244140625) and _rn16(_rn32(exact)) == Fraction(0.25)
    q_op, khat = _one_term([d], 64)
    s2 = attention.scores_hif4(q_op, np.array([[4.0]]), khat, 64)
    assert s2.dtype == np.float16 and float(s2[0, 0]) == 0.25


def test_score_scale_multiplies_the_group_sum():
    """The softmax scale multiplies the accumulated score once; it is not
    folded into the query's block scale first.  Witness (D = 64): b = 1.25,
    d = 48.6416015625: the group term d*b/4 is exact, fp16(fp32(fp32(d*b/4) * c))
    = 2.740234375, whereas folding the scale (fp16(fp32(d * fp32(b/4 * c))))
    gives 2.7421875."""
    from fractions import Fraction
    d, b = 48.6416015625, 1.25
    c = Fraction(float(attention.score_scale(64)))
    assert _rn16(_rn32(_rn32(Fraction(d) * Fraction(b) / 4) * c)) == Fraction(2.740234375)
    assert _rn16(_rn32(Fraction(d) * _rn32(Fraction(b) / 4 * c))) == Fraction(2.7421875)
    q_op, khat = _one_term([d], 64)
    s2 = attention.scores_hif4(q_op, np.array([[b]]), khat, 64)
    assert float(s2[0, 0]) == 2.740234375


def test_group_terms_sum_in_fp32():
    """The group terms are added in fp32 (each addition rounded once) before
    the scale.  Witness (D = 128): t = (-19.95166015625, -0.5801534652709961),
    exact in fp32; fp16(fp32(fp32(t0 + t1) * c)) = -2.619140625, while the
    exact sum scaled and rounded the same way gives -2.6171875."""
    from fractions import Fraction
    t0, t1 = -19.95166015625, -0.5801534652709961
    c = Fraction(float(attention.score_scale(128)))
    assert _rn16(_rn32(_rn32(Fraction(t0) + Fraction(t1)) * c)) == Fraction(-2.619140625)
    assert _rn16(_rn32((Fraction(t0) + Fraction(t1)) * c)) == Fraction(-2.6171875)
    q_op, khat = _one_term([t0, t1], 128)
    s2 = attention.scores_hif4(q_op, np.array([[4.0, 4.0]]), khat, 128)
    assert float(s2[0, 0]) == -2.619140625


def test_group_terms_sum_left_to_right():
    """At D = 256 the four group terms are summed in contraction order,
    ((t0 + t1) + t2) + t3.  Witness: t = (18.738555908203125,
    -2.418212890625, -0.21242237091064453, -0.6583194732666016) gives
    S2 = 1.3935546875; a pairwise sum (t0 + t1) + (t2 + t3) and the reversed
    order both give 1.392578125, and so does the witness with its groups
    reversed."""
    from fractions import Fraction
    t = [18.738555908203125, -2.418212890625, -0.21242237091064453, -0.6583194732666016]
    c = Fraction(float(attention.score_scale(256)))
    f = [Fraction(x) for x in t]
    left = _rn32(_rn32(_rn32(f[0] + f[1]) + f[2]) + f[3])
    pair = _rn32(_rn32(f[0] + f[1]) + _rn32(f[2] + f[3]))
    assert _rn16(_rn32(left * c)) == Fraction(1.3935546875) and _rn16(_rn32(pair * c)) == Fraction(1.392578125)
    q_op, khat = _one_term(t, 256)
    ones = np.full((1, 4), 4.0)
    assert float(attention.scores_hif4(q_op, ones, khat, 256)[0, 0]) == 1.3935546875
    q_op, khat = _one_term(t[::-1], 256)
    assert float(attention.scores_hif4(q_op, ones, khat, 256)[0, 0]) == 1.392578125


def test_scores_on_quantized_operands_match_exact_rounding():
    """On real quantized rows the oracle's scores equal an exact-rational
    evaluation from the dequantized values themselves (the oracle works from
    the operand values and the bases instead): each group term summed
    exactly from the dequantized Q^ and K^ elements, fp32 sums in group
    order, one fp32 multiply by c, fp16."""
    from fractions import Fraction
    q, k, v, cu = small_case(heads_q=1, heads_kv=1, seqlens=(6,), seed=17, head_dim=128)
    qf = attention.quantize_rows(q[:, 0])
    qhat = qf["xhat"].reshape(6, 128)
    khat = attention.quantize_rows(k[:, 0])["xhat"].reshape(6, 128)
    q_op = attention.unit_operands(qf).reshape(6, 128)
    s2 = attention.scores_hif4(q_op, qf["scale"], khat, 128)
    c = Fraction(float(attention.score_scale(128)))
    for i in range(6):
        for j in range(6):
            acc = None
            for g in range(2):
                tg = sum(Fraction(float(a)) * Fraction(float(b))
                         for a, b in zip(qhat[i, 64 * g:64 * g + 64], khat[j, 64 * g:64 * g + 64]))
                acc = tg if acc is None else _rn32(acc + tg)
            assert Fraction(float(s2[i, j])) == _rn16(_rn32(acc * c)), (i, j)


@pytest.mark.parametrize("d", [64, 128, 256])
def test_scores_within_one_fp16_step_of_exact(d):
    """Against brute force: S2 is within one fp16 step of the real-number
    score (dequantized Q^ . dequantized K^) * log2(e)/sqrt(D); a transposed
    operand, a dropped group, a wrong base or a wrong scale is far outside."""
    q, k, v, cu = small_case(heads_q=1, heads_kv=1, seqlens=(40,), seed=23, head_dim=d)
    qf = attention.quantize_rows(q[:, 0])
    qhat = qf["xhat"].reshape(40, d)
    khat = attention.quantize_rows(k[:, 0])["xhat"].reshape(40, d)
    s2 = attention.scores_hif4(attention.unit_operands(qf).reshape(40, d), qf["scale"], khat, d).astype(np.float64)
    ref = qhat @ khat.T * (math.log2(math.e) / math.sqrt(d))
    step = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref), 2.0 ** -14))) - 10)
    assert np.all(np.abs(s2 - ref) <= step)
    assert np.abs(s2 - ref).max() > 0                 # the scores are rounded, not exact


def test_p_only_theorem1_and_constant_v():
    """P-only local operator (Q, K, V unquantized fp16, only P quantized): the
    setting of Theorem 1 itself.  One-block rows satisfy both closed forms
    against the fp16 softmax weights a_j = P16_j and the raw V rows; a
    constant V row is returned exactly under P-Reordering and scaled by
    1 + eps under the inconsistent normalizer."""
    q, k, v, cu = small_case(heads_q=1, heads_kv=1, seqlens=(64,), seed=12)
    con = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, operands="p_only", want_p=True)[(0, 0)]
    mis = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, operands="p_only", norm="inconsistent")[(0, 0)]
    s2 = attention.scores_fp16(q[:, 0], k[:, 0], 128)
    vrows = v[:, 0].astype(np.float64)
    checked = 0
    for i in range(8, 64):
        keys = np.arange(i + 1)
        a = attention.exp2_fp16(attention.sub_fp16(s2[i, keys], s2[i, keys].max())).astype(np.float64)
        ahat = hif4.dequantize(hif4.unpack(con["p_codes"][i, 0], con["p_meta"][i, 0]))[: i + 1]
        nz = a > 0
        ostar, ebar, delta, w, e_t = _thm1_terms(a[nz], ahat[nz], vrows[keys][nz])
        tol = 1e-12 * (1 + np.abs(ostar).max())
        assert np.max(np.abs((con["o"][i] - ostar) - e_t / (1 + ebar))) < tol
        assert np.max(np.abs((mis["o"][i] - ostar) - (e_t + ebar * ostar))) < tol
        checked += 1
    assert checked > 40
    q, k, v, cu = small_case(heads_q=2, heads_kv=1, seqlens=(200,), seed=13)
    v[:] = v[3, 0]
    pre = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, operands="p_only")
    mis = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, operands="p_only", norm="inconsistent")
    for key in pre:
        assert np.array_equal(pre[key]["o16"], np.broadcast_to(v[3, 0], pre[key]["o16"].shape))
        ratio = pre[key]["l_con"] / pre[key]["l_mis"]
        assert np.allclose(mis[key]["o"], ratio[:, None] * v[3, 0].astype(np.float64)[None, :], rtol=1e-12)
        assert np.sum(np.abs(ratio - 1) > 1e-6) > 50
