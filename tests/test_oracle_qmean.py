"""Pins for the oracle's Q-Mean auxiliary (Algorithm 1, mu step and score
correction; Section 4.6; Appendix C).

  * the mean is the exact channel sum rounded once to fp16: a row whose exact
    mean lies just above an fp16 rounding midpoint, by less than an fp32 ulp,
    must round up (an fp32 accumulation would tie and round to even);
  * the key sums are exact before the fp32 rounding: 2048 plus 64 values of
    2^-13 is 2048 + 2^-7 (sequential fp32 additions would stay at 2048);
  * constant rows have mean equal to the constant and a zero Q_z; a shift of
    every query element by a constant leaves the Q_z codes unchanged;
  * the correction mu*kappa is added to the fp32 score accumulator after the
    group terms with one rounding, and scaled with the rest of the score;
  * with exact arithmetic the corrected scores equal the uncorrected ones,
    so the forward equals brute-force softmax attention;
  * on queries with a DC bias (the case Q-Mean exists for), the quantized
    forward with Q-Mean is much closer to exact attention than without it,
    and a sign, scale or dropped-term mistake in the correction is not."""
import numpy as np
import pytest

from oracle import attention, qmean
from paper_2607_04302_amd.workloads import small_case
from tests.test_oracle_attention import _brute


def test_mean_rounds_once_from_the_exact_sum():
    row = np.ones(128, np.float16)
    row[0] = np.float16(2.0625)
    row[1] = np.float16(2.0 ** -20)
    # exact mean = 1 + 2^-11 + 2^-27: above the midpoint of 1 and 1 + 2^-10
    mu = qmean.token_mean(row[None, :])
    assert mu.dtype == np.float16
    assert float(mu[0]) == 1.0 + 2.0 ** -10


def test_mean_of_known_rows():
    x = np.zeros((3, 64), np.float16)
    x[0, 5] = np.float16(3.0)                    # 3/64
    x[1] = np.float16(-0.75)                     # constant row
    x[2, ::2] = np.float16(1.0)
    x[2, 1::2] = np.float16(-1.0)                # zero mean
    mu = qmean.token_mean(x)
    assert list(mu.astype(np.float64)) == [3.0 / 64, -0.75, 0.0]
    z = qmean.zero_mean(x, mu)
    assert np.all(z[1] == 0)
    assert np.array_equal(z[2], x[2])
    assert float(z[0, 5]) == np.float16(3.0 - 3.0 / 64)


def test_key_sum_is_exact_before_rounding():
    k = np.zeros((1, 128), np.float16)
    k[0, 0] = np.float16(2048.0)
    k[0, 1:65] = np.float16(2.0 ** -13)
    kap = qmean.key_sums(k)
    assert kap.dtype == np.float32
    assert float(kap[0]) == 2048.0 + 2.0 ** -7


def test_correction_product_is_added_with_one_rounding():
    """fp32(acc + mu*kappa): the exact product enters the sum.  mu = 1 + 2^-10,
    kappa = 1 + 2^-23, acc = -1: the exact result 2^-10 + 2^-23 + 2^-33 is
    representable up to the last term (one rounding keeps 2^-23), while
    rounding the product first loses it."""
    mu = np.array([np.float16(1.0 + 2.0 ** -10)], np.float16)
    kap = np.array([np.float32(1.0 + 2.0 ** -23)], np.float32)
    acc = np.array([[np.float32(-1.0)]], np.float32)
    got = qmean.add_correction(acc, mu, kap)
    assert got.dtype == np.float32
    assert float(got[0, 0]) == 2.0 ** -10 + 2.0 ** -23 + 2.0 ** -33
    assert float(np.float32(np.float32(float(mu[0]) * float(kap[0])) - 1.0)) == 2.0 ** -10 + 2.0 ** -23


def test_correction_follows_the_group_terms_and_takes_the_scale():
    """S2 = fp16(fp32(fp32(fp32(t0 + t1) + mu*kappa) * c)): the correction is
    added after the group terms, before the scale.  Witness (D = 128):
    t = (0.7456512451171875, 14.5777587890625), mu = -2.99609375,
    kappa = -38.7888298034668 give 16.765625; adding a rounded product, or
    adding the correction before the group terms, gives 16.78125."""
    from fractions import Fraction
    from tests.test_oracle_attention import _one_term, _rn16, _rn32
    t0, t1, mu, kap = 0.7456512451171875, 14.5777587890625, -2.99609375, -38.7888298034668
    c = Fraction(float(attention.score_scale(128)))
    f0, f1, fm, fk = Fraction(t0), Fraction(t1), Fraction(mu), Fraction(float(np.float32(kap)))
    assert _rn16(_rn32(_rn32(_rn32(f0 + f1) + fm * fk) * c)) == Fraction(16.765625)
    assert _rn16(_rn32(_rn32(_rn32(f0 + f1) + _rn32(fm * fk)) * c)) == Fraction(16.78125)
    assert _rn16(_rn32(_rn32(_rn32(fm * fk + f0) + f1) * c)) == Fraction(16.78125)
    q_op, khat = _one_term([t0, t1], 128)
    s2 = attention.scores_hif4(q_op, np.array([[4.0, 4.0]]), khat, 128,
                               corr=(np.array([mu], np.float16), np.array([kap], np.float32)))
    assert float(s2[0, 0]) == 16.765625


def test_dc_shift_leaves_q_codes_unchanged():
    rng = np.random.default_rng(3)
    q = rng.integers(-6, 7, size=(5, 2, 128)).astype(np.float16)   # exact means
    k = rng.standard_normal((5, 1, 128)).astype(np.float16)
    mu0, kap0, c0, m0 = attention.quantize_q_mean(q, k)
    mu1, kap1, c1, m1 = attention.quantize_q_mean((q.astype(np.float32) + 2.0).astype(np.float16), k)
    assert np.array_equal(c0, c1) and np.array_equal(m0, m1)
    assert np.array_equal(mu1.astype(np.float64), mu0.astype(np.float64) + 2.0)
    assert np.array_equal(kap0, kap1)


@pytest.mark.parametrize("lens", [(1,), (65,), (130, 17)])
def test_exact_mode_with_q_mean_equals_softmax_attention(lens):
    q, k, v, cu = small_case(heads_q=4, heads_kv=2, seqlens=lens, seed=13, q_bias=2.0)
    ref = _brute(q, k, v, cu, 2)
    res = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, arith="exact", q_mean=True)
    for (b, h), r in res.items():
        want = ref[cu[b]:cu[b + 1], h]
        assert np.max(np.abs(r["o"] - want)) < 1e-12 * max(1.0, np.abs(want).max())


def _rel(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def test_q_mean_removes_the_dc_bias_error(monkeypatch):
    q, k, v, cu = small_case(heads_q=2, heads_kv=1, seqlens=(256,), seed=5, q_bias=3.0)
    ex = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, arith="exact")
    plain = attention.attention_fwd(q, k, v, None, cu_seqlens=cu)
    qm = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, q_mean=True)
    for key in ex:
        e_plain, e_qm = _rel(plain[key]["o"], ex[key]["o"]), _rel(qm[key]["o"], ex[key]["o"])
        assert e_qm < 0.2 and e_qm < 0.7 * e_plain, (key, e_qm, e_plain)
    # the same check fails for a planted sign or scale mistake in the correction
    good = qmean.add_correction
    for bad in (lambda acc, mu, ka: good(acc, -mu, ka),
                lambda acc, mu, ka: good(acc, mu, ka * np.float32(0.5))):
        monkeypatch.setattr(qmean, "add_correction", bad)
        wrong = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, q_mean=True)
        assert min(_rel(wrong[key]["o"], ex[key]["o"]) for key in ex) > 0.3
