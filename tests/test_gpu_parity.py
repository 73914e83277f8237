"""GPU parity: the HIP path against the CPU oracle on the same seeded inputs.

Bit-exact: the kernels' fp16 exponential (all inputs), Q^/K^/V^ codes and
metadata, and every P^ group written by the attention kernel's debug dump.
Tolerance (element-wise |gpu - ref| <= 2e-3 + 1e-2*|ref|): O and LSE."""
import sys

import numpy as np
import pytest

from oracle import attention as oatt
from oracle import hif4 as ohif4
from oracle import smooth as osmooth
from oracle.softmax16 import exp2_fp16
from paper_2607_04302_amd.workloads import WORKLOADS, make_calibration, make_inputs, small_case

from _edge import edge_rows, edge_tokens
from _jump import check_jumps, jump_case
from _gpu_util import check_close, to_gpu, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def h():
    import paper_2607_04302_amd as mod
    mod.load_library()
    return mod


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def test_exp2_exhaustive(h):
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    x = bits.view(np.float16)
    sel = (np.isfinite(x) & (x <= 0)) | (x == -np.inf)
    xs = x[sel]
    got = to_np(h.hifa4_selftest_exp2(to_gpu(xs)))
    want = exp2_fp16(xs)
    assert np.array_equal(got.view(np.uint16), want.view(np.uint16))


@pytest.mark.parametrize("d,hq,hkv,lens", [(128, 4, 2, (200,)), (64, 2, 2, (77, 130)), (256, 2, 1, (96,))])
def test_quantize_qk_bitexact(h, d, hq, hkv, lens):
    q, k, v, cu = small_case(heads_q=hq, heads_kv=hkv, head_dim=d, seqlens=lens, seed=d + hq)
    s = np.exp(np.random.default_rng(1).uniform(-2, 2, (hkv, d))).astype(np.float32)
    for sv in (None, s):
        qc, qm, kc, km = oatt.quantize_qk(q, k, sv)
        cu_t = to_gpu(cu)
        g = h.hifa4_quantize_qk(to_gpu(q), to_gpu(k), None if sv is None else to_gpu(sv),
                                cu_seqlens=cu_t, max_seqlen=max(lens))
        assert np.array_equal(to_np(g[0]), qc)
        assert np.array_equal(to_np(g[1]).view(np.uint32), qm)
        assert np.array_equal(to_np(g[2]), kc)
        assert np.array_equal(to_np(g[3]).view(np.uint32), km)


@pytest.mark.parametrize("d", [64, 128, 256])
def test_quantize_edge_values_bitexact(h, d):
    """Q^, K^ and V^ codes and metadata of inputs built from the quantizer's
    special cases (zero groups, one element, rounding ties, subnormals, large
    magnitudes, nested E2/E3 blocks, negative zeros), with and without
    smoothing."""
    lens = (130, 64, 1, 77)
    q, k, v, cu = small_case(heads_q=4, heads_kv=2, head_dim=d, seqlens=lens, seed=31)
    edge_rows(q, 31)
    edge_rows(k, 32)
    edge_tokens(v, cu, 33)
    s = np.exp(np.random.default_rng(34).uniform(-2, 2, (2, d))).astype(np.float32)
    for sv in (None, s):
        qc, qm, kc, km = oatt.quantize_qk(q, k, sv)
        g = h.hifa4_quantize_qk(to_gpu(q), to_gpu(k), None if sv is None else to_gpu(sv),
                                cu_seqlens=to_gpu(cu), max_seqlen=max(lens))
        assert np.array_equal(to_np(g[0]), qc)
        assert np.array_equal(to_np(g[1]).view(np.uint32), qm)
        assert np.array_equal(to_np(g[2]), kc)
        assert np.array_equal(to_np(g[3]).view(np.uint32), km)
    nb = -(-max(lens) // 64)
    gv = h.hifa4_quantize_v(to_gpu(v), cu_seqlens=to_gpu(cu), max_seqlen=max(lens))
    codes, meta = _canon_v_padded(v, cu, nb)
    assert np.array_equal(to_np(gv[0]), codes)
    assert np.array_equal(to_np(gv[1]).view(np.uint32), meta)


def _canon_v_padded(v, cu, nb):
    """Oracle V^ codes in the padded [B, NB, Hkv, D] layout."""
    hkv, d = v.shape[1], v.shape[2]
    codes = np.zeros((len(cu) - 1, nb, hkv, d, 32), np.uint8)
    meta = np.zeros((len(cu) - 1, nb, hkv, d), np.uint32)
    for b in range(len(cu) - 1):
        for hk in range(hkv):
            f, _ = oatt.quantize_tokens(v[cu[b]:cu[b + 1], hk])        # [D, G_b, 64]
            c_, m_ = ohif4.pack(f)
            gb = c_.shape[1]
            codes[b, :gb, hk] = c_.transpose(1, 0, 2)
            meta[b, :gb, hk] = m_.T
        # groups past the end are all-zero groups
        zc, zm = ohif4.pack(ohif4.quantize(np.zeros(64)))
        gb = -(-(cu[b + 1] - cu[b]) // 64)
        codes[b, gb:] = zc
        meta[b, gb:] = zm
    return codes, meta


def test_quantize_v_bitexact(h):
    q, k, v, cu = small_case(heads_q=2, heads_kv=2, head_dim=128, seqlens=(200, 64, 1, 129), seed=3)
    nb = -(-200 // 64)
    g = h.hifa4_quantize_v(to_gpu(v), cu_seqlens=to_gpu(cu), max_seqlen=200)
    codes, meta = _canon_v_padded(v, cu, nb)
    assert np.array_equal(to_np(g[0]), codes)
    assert np.array_equal(to_np(g[1]).view(np.uint32), meta)


def _run_and_compare(h, q, k, v, cu, s, max_seqlen, norm="preorder", heads=None, rows=None, check_p=True,
                     seqs=None, q_mean=False, dump_per_head=False):
    """Runs the HIP forward on the whole problem, the oracle on the sampled
    (sequence, head, row) set, and compares O, LSE and (check_p) the P^ dump.
    Only the sampled slices of the GPU outputs are copied to the host.
    dump_per_head: the P^ dump is taken head by head (a dump window of one
    query head, one more forward per sampled head), for problems whose whole
    dump would not fit."""
    import torch
    cu_t = None if cu is None else to_gpu(cu)
    nm = h.NORM_PREORDER if norm == "preorder" else h.NORM_INCONSISTENT
    args = (to_gpu(q), to_gpu(k), to_gpu(v), None if s is None else to_gpu(s))
    res = h.hifa4_attention_fwd(*args, cu_seqlens=cu_t, max_seqlen=max_seqlen, norm=nm,
                                debug_p=check_p and not dump_per_head, q_mean=q_mean)
    o, lse = res[0], res[1]
    dumps = {}
    if check_p and dump_per_head:
        for hh in heads:
            r1 = h.hifa4_attention_fwd(*args, cu_seqlens=cu_t, max_seqlen=max_seqlen, norm=nm, debug_p=True,
                                       q_mean=q_mean, debug_heads=(hh, 1))
            dumps[hh] = (r1[2][0], r1[3][0])
            torch.cuda.synchronize()
    elif check_p:
        dumps = {hh: (res[2][hh], res[3][hh]) for hh in range(q.shape[-2])}
    ref = oatt.attention_fwd(q, k, v, s, cu_seqlens=cu, norm=norm, heads=heads, rows=rows, want_p=check_p,
                             seqs=seqs, q_mean=q_mean)
    if cu is None:
        bsz, S = q.shape[:2]
        cuv = np.arange(bsz + 1) * S
        o = o.reshape(bsz * S, *o.shape[2:])
    else:
        cuv = cu
    worst = 0.0
    for (b, hh), r in ref.items():
        if len(r["rows"]) == 0:
            continue                                # an empty sequence has no rows
        tok = cuv[b] + r["rows"]
        tok_t = torch.as_tensor(tok, device=o.device, dtype=torch.long)
        worst = max(worst, check_close(to_np(o[tok_t, hh]), r["o"], what=f"O seq {b} head {hh}"))
        check_close(to_np(lse[hh, tok_t]), r["lse"], atol=2e-3, rtol=0, what="LSE")
        if check_p:
            pc = to_np(dumps[hh][0][tok_t])
            pm = to_np(dumps[hh][1][tok_t]).view(np.uint32)
            for ii, i in enumerate(r["rows"]):
                nb_i = i // 64 + 1
                assert np.array_equal(pc[ii, :nb_i], r["p_codes"][ii, :nb_i]), (b, hh, i)
                assert np.array_equal(pm[ii, :nb_i], r["p_meta"][ii, :nb_i]), (b, hh, i)
    return worst


def test_tiny_config_full_parity(h):
    """The tiny causal prefill workload (S=256, D=128) with Smooth-QK scales
    from its 4-sequence calibration draw: every P^ code bit-exact, O, LSE."""
    w = WORKLOADS["tiny_s256"]
    q, k, v, _ = make_inputs(w)
    qc, kc = make_calibration(w)
    s, _ = osmooth.calibrate(qc, kc, w.heads_kv, w.alpha)
    _say("tiny_s256 preorder")
    err = _run_and_compare(h, q, k, v, None, s, w.seqlen)
    _say("tiny_s256 max err", err)
    _say("tiny_s256 inconsistent")
    _run_and_compare(h, q, k, v, None, s, w.seqlen, norm="inconsistent")


@pytest.mark.parametrize("d,hq,hkv,lens,seed", [
    (128, 4, 1, (300, 65, 64, 1, 190), 1),      # GQA x4, ragged tails, single token
    (128, 4, 2, (0, 130, 0, 65), 4),             # empty sequences between others
    (64, 2, 2, (129, 511), 2),                   # no GQA, D=64
    (256, 4, 2, (200, 33), 3),                   # GQA x2, D=256
    (128, 8, 8, (97,), 4),
    (128, 16, 2, (150, 70), 6),                 # GQA x8: two workgroups of four heads per kv head
    (64, 6, 2, (100, 33), 7),                    # GQA x3: one head per workgroup, 128-row tiles
])
def test_varlen_parity(h, d, hq, hkv, lens, seed):
    q, k, v, cu = small_case(heads_q=hq, heads_kv=hkv, head_dim=d, seqlens=lens, seed=seed)
    s = np.exp(np.random.default_rng(seed).uniform(-1, 1.5, (hkv, d))).astype(np.float32)
    _say("varlen", d, hq, hkv, lens)
    _run_and_compare(h, q, k, v, cu, s, max(lens))
    _run_and_compare(h, q, k, v, cu, None, max(lens), norm="inconsistent")


@pytest.mark.parametrize("d,hq,hkv,smooth", [(128, 4, 2, False), (64, 2, 1, True), (256, 2, 1, False)])
def test_edge_values_parity(h, d, hq, hkv, smooth):
    """The attention kernel's own quantizers (Q in its prologue, K and V in
    the pre-pass) on inputs built from the quantizer's special cases: every
    P^ code bit-exact, O and LSE within tolerance.  Magnitudes stay below 40
    so that no score leaves the fp16 range."""
    lens = (200, 77)
    q, k, v, cu = small_case(heads_q=hq, heads_kv=hkv, head_dim=d, seqlens=lens, seed=41)
    edge_rows(q, 41, large=40.0)
    edge_rows(k, 42, large=40.0)
    edge_tokens(v, cu, 43, large=40.0)
    s = np.exp(np.random.default_rng(44).uniform(-1, 1, (hkv, d))).astype(np.float32) if smooth else None
    _say("edge values", d, hq, hkv, smooth)
    _run_and_compare(h, q, k, v, cu, s, max(lens))


def test_fp16_variant(h):
    for d in (64, 128, 256):
        q, k, v, cu = small_case(heads_q=4, heads_kv=2, head_dim=d, seqlens=(300, 47), seed=9)
        _say("fp16 variant D", d)
        o, lse = h.hifa4_attention_fwd(to_gpu(q), to_gpu(k), to_gpu(v), None, cu_seqlens=to_gpu(cu),
                                       max_seqlen=300, operands=h.OPERANDS_FP16)
        o, lse = to_np(o), to_np(lse)
        ref = oatt.attention_fwd(q, k, v, None, cu_seqlens=cu, operands="fp16")
        for (b, hh), r in ref.items():
            tok = cu[b] + r["rows"]
            # The FP16 reference sums q.k in fp32 in the MFMA's own order, so a
            # score can round to the neighbouring fp16 value (one ulp: 2^-11
            # relative); that scales one weight by 2^(2^-7) ~ 1.0054 at
            # |S2| < 16 and moves O by up to 0.54% of |v - O| for that key, and
            # LSE by up to ulp(m)*ln2 ~ 1e-3*|LSE|.
            check_close(o[tok, hh], r["o"], atol=1e-2, rtol=1e-2, what="fp16 O")
            check_close(lse[hh, tok], r["lse"], atol=2e-3, rtol=1e-3, what="fp16 LSE")


def test_constant_v_invariant(h):
    """A constant V row comes back bit-exactly under P-Reordering; the
    inconsistent normalizer scales it by (1 + eps) (Theorem 1 with e_t = 0)."""
    q, k, v, cu = small_case(heads_q=2, heads_kv=1, head_dim=128, seqlens=(333,), seed=9)
    v[:] = v[0, 0]
    _, vhat = oatt.quantize_tokens(v[:, 0])
    target = vhat[0].astype(np.float16)
    o, _ = h.hifa4_attention_fwd(to_gpu(q), to_gpu(k), to_gpu(v), None, cu_seqlens=to_gpu(cu), max_seqlen=333)
    o = to_np(o)
    assert np.array_equal(o, np.broadcast_to(target, o.shape))
    om, _ = h.hifa4_attention_fwd(to_gpu(q), to_gpu(k), to_gpu(v), None, cu_seqlens=to_gpu(cu), max_seqlen=333,
                                  norm=h.NORM_INCONSISTENT)
    om = to_np(om)
    assert (om != np.broadcast_to(target, om.shape)).mean() > 0.5


def test_calibration(h):
    w = WORKLOADS["tiny_s256"]
    qc, kc = make_calibration(w)
    for alpha in (0.5, 0.25, 0.0, -1.0):
        s_ref, rep = osmooth.calibrate(qc, kc, w.heads_kv, alpha)
        s_gpu, grep = h.hifa4_calibrate_smooth_qk(to_gpu(qc), to_gpu(kc), alpha)
        s_gpu = to_np(s_gpu)
        # same float64 formulas on both sides; allow one fp32 ulp for libm pow
        ulp = np.abs(s_gpu.view(np.int32).astype(np.int64) - s_ref.view(np.int32).astype(np.int64))
        assert ulp.max() <= 1, alpha
        assert abs(grep["rho_k"] - rep["rho_k"]) < 1e-9 * rep["rho_k"]
        assert abs(grep["t_kq"] - rep["t_kq"]) < 1e-12 * rep["t_kq"]
        assert grep["branch"] == rep["branch"]


def test_qwen3_shape_sampled(h):
    """Qwen3-8B-shaped S=4096 workload at full size, in the launch the
    benchmark times: sampled heads (one per KV group plus neighbours) and
    rows spanning the first, middle and last blocks, P^ codes bit-exact."""
    w = WORKLOADS["qwen3_8b_s4096"]
    q, k, v, _ = make_inputs(w)
    qc, kc = make_calibration(w, n=4)
    s, _ = osmooth.calibrate(qc, kc, w.heads_kv, w.alpha)
    rows = [0, 1, 31, 63, 64, 65, 1000, 2047, 2048, 3071, 4031, 4094, 4095]
    _say("qwen3 sampled")
    _run_and_compare(h, q, k, v, None, s, w.seqlen, heads=[0, 3, 4, 17, 31], rows=rows)


def test_long_s32768_sampled(h):
    """Long prefill, S=32768, at full size in the benchmark's launch shape,
    Smooth-QK scales from the Qwen3-shaped calibration draw: sampled heads and
    rows (first, block edges, middle, last); every P^ code of those rows bit
    exact (a dump window of one head at a time: 0.5 GiB instead of 17 GB for
    every head), O and LSE against the oracle."""
    w = WORKLOADS["long_s32768"]
    q, k, v, _ = make_inputs(w)
    qc, kc = make_calibration(WORKLOADS[w.calib_from], n=4)
    s, _ = osmooth.calibrate(qc, kc, w.heads_kv, w.alpha)
    rows = [0, 63, 64, 4097, 16383, 16384, 32700, 32767]
    _say("long_s32768 sampled")
    _run_and_compare(h, q, k, v, None, s, w.seqlen, heads=[2, 29], rows=rows, dump_per_head=True)


def test_varlen_b16_full(h):
    """Batched variable-length prefill (16 sequences of 512..2048 tokens,
    packed with cu_seqlens, Smooth-QK off) at full size: every sequence,
    sampled heads and rows, P^ codes bit-exact; then the inconsistent
    normalizer on the same inputs."""
    w = WORKLOADS["varlen_b16"]
    q, k, v, cu = make_inputs(w)
    rows = [0, 1, 63, 64, 300, 511, 1000, 1500, 2047]
    _say("varlen_b16 preorder")
    _run_and_compare(h, q, k, v, cu, None, int(w.seqlens().max()), heads=[0, 13, 31], rows=rows)
    _say("varlen_b16 inconsistent")
    _run_and_compare(h, q, k, v, cu, None, int(w.seqlens().max()), norm="inconsistent", heads=[5], rows=rows,
                     check_p=False)


def test_wide_d256_sampled(h):
    """Wide heads (D=256, B=2, S=8192, Smooth-QK on) at full size: sampled
    sequences, heads and rows, P^ codes bit-exact; the inconsistent
    normalizer's O and LSE against the oracle's."""
    w = WORKLOADS["wide_d256"]
    q, k, v, _ = make_inputs(w)
    qc, kc = make_calibration(w, n=2, seqlen=2048)
    s, _ = osmooth.calibrate(qc, kc, w.heads_kv, w.alpha)
    rows = [0, 64, 2047, 4096, 8191]
    _say("wide_d256 preorder")
    _run_and_compare(h, q, k, v, None, s, w.seqlen, heads=[1, 14], rows=rows, seqs=[0, 1])
    _say("wide_d256 inconsistent")
    _run_and_compare(h, q, k, v, None, s, w.seqlen, norm="inconsistent", heads=[6], rows=rows, seqs=[1],
                     check_p=False)


# ---------------------------------------------------------------------------
# Q-Mean auxiliary (Algorithm 1, the mean step and the score correction).
# mu, Q_z and the key sums kappa enter every score, so bit-exact P^ codes on
# every row check all three against the oracle's definitions.

def test_qmean_tiny_full_parity(h):
    w = WORKLOADS["tiny_s256"]
    q, k, v, _ = make_inputs(w)
    qc, kc = make_calibration(w)
    s, _ = osmooth.calibrate(qc, kc, w.heads_kv, w.alpha)
    _say("tiny_s256 q_mean")
    _run_and_compare(h, q, k, v, None, s, w.seqlen, q_mean=True)


@pytest.mark.parametrize("d,hq,hkv,lens,seed,bias", [
    (128, 4, 1, (300, 65, 64, 1, 190), 1, 2.0),   # DC-biased queries, GQA x4, ragged tails
    (64, 2, 2, (129, 511), 2, -1.5),               # D=64
    (256, 4, 2, (200, 33), 3, 0.75),               # D=256
    (128, 8, 8, (97,), 4, 0.0),                    # no bias: mu near zero
])
def test_qmean_varlen_parity(h, d, hq, hkv, lens, seed, bias):
    q, k, v, cu = small_case(heads_q=hq, heads_kv=hkv, head_dim=d, seqlens=lens, seed=seed, q_bias=bias)
    s = np.exp(np.random.default_rng(seed).uniform(-1, 1.5, (hkv, d))).astype(np.float32)
    _say("q_mean varlen", d, hq, hkv, lens, bias)
    _run_and_compare(h, q, k, v, cu, s, max(lens), q_mean=True)
    _run_and_compare(h, q, k, v, cu, None, max(lens), norm="inconsistent", q_mean=True)


def test_qmean_qwen3_shape_sampled(h):
    """Q-Mean on the Qwen3-8B-shaped S=4096 workload, full size, sampled heads
    and rows, P^ codes bit-exact."""
    w = WORKLOADS["qwen3_8b_s4096"]
    q, k, v, _ = make_inputs(w)
    qc, kc = make_calibration(w, n=4)
    s, _ = osmooth.calibrate(qc, kc, w.heads_kv, w.alpha)
    rows = [0, 1, 63, 64, 2047, 4031, 4095]
    _say("qwen3 sampled q_mean")
    _run_and_compare(h, q, k, v, None, s, w.seqlen, heads=[0, 5, 31], rows=rows, q_mean=True)


# ---------------------------------------------------------------------------
# P-only local operator (Q, K, V fp16; only P quantized).  Its scores are fp32
# sums in the MFMA's own order, so P^ codes are compared bit for bit on
# integer-valued Q and K, where every partial sum is exact in fp32 and the
# scores agree exactly with the oracle's; Gaussian inputs are checked
# statistically (a score one fp16 ulp off can move one P^ code by one step).

def _int_case(hq, hkv, d, lens, seed):
    rng = np.random.default_rng(seed)
    t = int(sum(lens))
    q = rng.integers(-1, 2, size=(t, hq, d)).astype(np.float16)
    k = rng.integers(-1, 2, size=(t, hkv, d)).astype(np.float16)
    v = rng.standard_normal((t, hkv, d)).astype(np.float32).astype(np.float16)
    return q, k, v, np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)


def _run_ponly(h, q, k, v, cu, max_seqlen, norm, debug_p):
    nm = h.NORM_PREORDER if norm == "preorder" else h.NORM_INCONSISTENT
    return h.hifa4_attention_fwd(to_gpu(q), to_gpu(k), to_gpu(v), None, cu_seqlens=to_gpu(cu), max_seqlen=max_seqlen,
                                 norm=nm, operands=h.OPERANDS_P_ONLY, debug_p=debug_p)


@pytest.mark.parametrize("d,hq,hkv,lens", [(128, 4, 1, (300, 65, 1)), (64, 2, 2, (129, 200)), (256, 4, 2, (150,))])
def test_p_only_exact_scores(h, d, hq, hkv, lens):
    q, k, v, cu = _int_case(hq, hkv, d, lens, seed=d + hq)
    for norm in ("preorder", "inconsistent"):
        _say("p_only exact scores", d, hq, hkv, lens, norm)
        res = _run_ponly(h, q, k, v, cu, max(lens), norm, True)
        ref = oatt.attention_fwd(q, k, v, None, cu_seqlens=cu, operands="p_only", norm=norm, want_p=True)
        o, lse = to_np(res[0]), to_np(res[1])
        pc, pm = to_np(res[2]), to_np(res[3]).view(np.uint32)
        for (b, hh), r in ref.items():
            tok = cu[b] + r["rows"]
            check_close(o[tok, hh], r["o"], what=f"p_only O seq {b} head {hh}")
            check_close(lse[hh, tok], r["lse"], atol=2e-3, rtol=0, what="p_only LSE")
            for ii, i in enumerate(r["rows"]):
                nb_i = i // 64 + 1
                assert np.array_equal(pc[hh, tok[ii], :nb_i], r["p_codes"][ii, :nb_i]), (b, hh, i)
                assert np.array_equal(pm[hh, tok[ii], :nb_i], r["p_meta"][ii, :nb_i]), (b, hh, i)


def test_p_only_gaussian(h):
    q, k, v, cu = small_case(heads_q=4, heads_kv=2, head_dim=128, seqlens=(400, 77), seed=21)
    for norm in ("preorder", "inconsistent"):
        o, lse = _run_ponly(h, q, k, v, cu, 400, norm, False)
        o, lse = to_np(o).astype(np.float64), to_np(lse)
        ref = oatt.attention_fwd(q, k, v, None, cu_seqlens=cu, operands="p_only", norm=norm)
        for (b, hh), r in ref.items():
            tok = cu[b] + r["rows"]
            g, w = o[tok, hh], r["o"]
            cos = (g * w).sum(1) / (np.linalg.norm(g, axis=1) * np.linalg.norm(w, axis=1))
            assert cos.min() > 0.999, (norm, b, hh, cos.min())
            assert np.mean(np.abs(g - w) <= 2e-3 + 1e-2 * np.abs(w)) > 0.99
            check_close(lse[hh, tok], r["lse"], atol=5e-3, rtol=1e-3, what="p_only LSE")


def _calib_layer(rng, k_sigma, q_sigma, outlier, n=4, S=256, hq=4, hkv=1, d=128):
    q = (rng.standard_normal((n, S, hq, d)) * q_sigma).astype(np.float16)
    k = rng.standard_normal((n, S, hkv, d)) * k_sigma
    if outlier:
        k[..., 7] *= outlier          # one channel of 128: under 1% of K's elements
    return q, k.astype(np.float16)


def test_calibration_layers(h):
    """Per-layer calibration in one call (the gate decides per layer): three
    layers built so that the literal gate picks Strong (one x12 outlier
    channel, T ~ 7), Mild (the same outlier with a wider Q, T ~ 2.7) and
    Bypass (no outlier); every layer's scales and report equal the oracle's
    single-layer calibration."""
    rng = np.random.default_rng(77)
    layers = [_calib_layer(rng, 1.0, 1.0, 12.0), _calib_layer(rng, 0.1, 0.35, 12.0), _calib_layer(rng, 1.0, 1.0, 0)]
    qs = np.stack([l[0] for l in layers])
    ks = np.stack([l[1] for l in layers])
    s_gpu, reps = h.hifa4_calibrate_smooth_qk_layers(to_gpu(qs), to_gpu(ks), -1.0)
    s_gpu = to_np(s_gpu)
    branches = []
    for i, (q, k) in enumerate(layers):
        s_ref, rep = osmooth.calibrate(q, k, 1, -1.0)
        ulp = np.abs(s_gpu[i].view(np.int32).astype(np.int64) - s_ref.view(np.int32).astype(np.int64))
        assert ulp.max() <= 1, i
        assert reps[i]["branch"] == rep["branch"], i
        assert abs(reps[i]["rho_k"] - rep["rho_k"]) < 1e-9 * rep["rho_k"]
        assert abs(reps[i]["t_kq"] - rep["t_kq"]) < 1e-12 * rep["t_kq"]
        branches.append(rep["branch"])
    assert branches == [2, 1, 0]


# ---------------------------------------------------------------------------
# The running maximum's special paths ("P-Reordering under online softmax"):
# a block whose maximum exceeds the running maximum by more than 25 in log2
# units makes the rescale factor r = E(fp16(m - m_new)) exactly 0 (the
# history is wiped), and a maximum that grows in steps below that over more
# than 64 units drives the product of the rescale factors below 2^-64, where
# the kernel's deferred rescale renormalizes.  Integer Q and K keep the fp16
# scores exact on the P-only path too, so P^ is bit-exact there as well.

@pytest.mark.parametrize("kind", ["wipe", "renorm"])
@pytest.mark.parametrize("d,hq,hkv", [(128, 2, 1), (64, 4, 2)])
def test_running_max_special_paths(h, kind, d, hq, hkv):
    lens = (450, 200)
    q, k, v, cu = jump_case(kind, lens, hq, hkv, d, seed=61 + d)
    check_jumps(kind, q, k, cu, d, "hif4")
    for norm in ("preorder", "inconsistent"):
        _say("running max", kind, d, hq, hkv, norm)
        _run_and_compare(h, q, k, v, cu, None, max(lens), norm=norm)


@pytest.mark.parametrize("kind", ["wipe", "renorm"])
def test_running_max_special_paths_p_only(h, kind):
    lens = (450, 130)
    d, hq, hkv = 128, 2, 1
    q, k, v, cu = jump_case(kind, lens, hq, hkv, d, seed=71)
    check_jumps(kind, q, k, cu, d, "p_only")
    for norm in ("preorder", "inconsistent"):
        _say("running max p_only", kind, norm)
        res = _run_ponly(h, q, k, v, cu, max(lens), norm, True)
        ref = oatt.attention_fwd(q, k, v, None, cu_seqlens=cu, operands="p_only", norm=norm, want_p=True)
        o, lse = to_np(res[0]), to_np(res[1])
        pc, pm = to_np(res[2]), to_np(res[3]).view(np.uint32)
        for (b, hh), r in ref.items():
            tok = cu[b] + r["rows"]
            check_close(o[tok, hh], r["o"], what=f"p_only O seq {b} head {hh}")
            check_close(lse[hh, tok], r["lse"], atol=2e-3, rtol=0, what="p_only LSE")
            for ii, i in enumerate(r["rows"]):
                nb_i = i // 64 + 1
                assert np.array_equal(pc[hh, tok[ii], :nb_i], r["p_codes"][ii, :nb_i]), (b, hh, i)
                assert np.array_equal(pm[hh, tok[ii], :nb_i], r["p_meta"][ii, :nb_i]), (b, hh, i)
