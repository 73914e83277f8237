"""Pins for the oracle's Q-Mean auxiliary (Algorithm 1, mu step and score
correction; Section 4.6; Appendix C).

  * the mean is the exact channel sum rounded once to fp16: a row whose exact
    mean lies just above an fp16 rounding midpoint, by less than an fp32 ulp,
    must round up (an fp32 accumulation would tie and round to even);
  * the key sums are exact before the fp32 rounding: 2048 plus 64 values of
    2^-13 is 2048 + 2^-7 (sequential fp32 additions would stay at 2048);
  * constant rows have mean equal to the constant and a zero Q_z; a shift of
    every query element by a constant leaves the Q_z codes unchanged;
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


def test_correction_product_rounds_once_to_fp32():
    mu = np.array([np.float16(1.0 + 2.0 ** -10)], np.float16)
    kap = np.array([np.float32(1.0 + 2.0 ** -23)], np.float32)
    # exact product 1 + 2^-10 + 2^-23 + 2^-33 rounds to 1 + 2^-10 + 2^-23
    c = qmean.correction(mu, kap, np.float32(1.0))
    assert c.dtype == np.float32
    assert float(c[0, 0]) == 1.0 + 2.0 ** -10 + 2.0 ** -23


def test_correction_scales_the_mean_first():
    """corr = fp32(fp32(mu*c) * kappa): mu*c is rounded to fp32 before the
    product with kappa.  Witness (D = 128, c = fp32(log2(e)/sqrt(128))):
    mu = -0.496826171875, kappa = 12.613357543945312 gives
    -0.7991066575050354; one rounding of the exact triple product would give
    -0.7991065979003906."""
    from fractions import Fraction
    from tests.test_oracle_attention import _rn32
    from oracle.attention import score_scale
    mu = np.array([np.float16(-0.496826171875)], np.float16)
    kap = np.array([np.float32(12.613357543945312)], np.float32)
    c = score_scale(128)
    got = Fraction(float(qmean.correction(mu, kap, c)[0, 0]))
    f_mu, f_c, f_k = Fraction(float(mu[0])), Fraction(float(c)), Fraction(float(kap[0]))
    assert got == _rn32(_rn32(f_mu * f_c) * f_k) == Fraction(-0.7991066575050354)
    assert _rn32(f_mu * f_c * f_k) == Fraction(-0.7991065979003906)


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
    good = attention.correction
    for bad in (lambda mu, ka, c: -good(mu, ka, c), lambda mu, ka, c: good(mu, ka, c) * np.float32(0.5)):
        monkeypatch.setattr(attention, "correction", bad)
        wrong = attention.attention_fwd(q, k, v, None, cu_seqlens=cu, q_mean=True)
        assert min(_rel(wrong[key]["o"], ex[key]["o"]) for key in ex) > 0.3
