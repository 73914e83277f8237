"""GPU parity of the decode step over a packed HIF4 cache.

The oracle needs no decode mode: a decode step is row L-1 of the causal
prefill of the cached sequence (the newest token sees every key).  For each
sampled (sequence, kv head) the oracle runs that single row on the
sequence's K and V with a query array whose last row is the decode query.
Bit-exact: every P^ group of the decode kernels' debug dump; tolerance
(|gpu - ref| <= 2e-3 + 1e-2*|ref|): O; LSE within 2e-3."""
import sys

import numpy as np
import pytest

from oracle import attention as oatt
from oracle import smooth as osmooth
from paper_2607_04302_amd.workloads import WORKLOADS, make_calibration, make_decode_inputs, small_case

from _edge import edge_rows
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


def _build_cache(h, k, v, s, cu, max_seqlen):
    cu_t = None if cu is None else to_gpu(cu)
    _, _, kc, km = h.hifa4_quantize_qk(None, to_gpu(k), None if s is None else to_gpu(s),
                                       cu_seqlens=cu_t, max_seqlen=max_seqlen)
    vc, vm = h.hifa4_quantize_v(to_gpu(v), cu_seqlens=cu_t, max_seqlen=max_seqlen)
    return kc, km, vc, vm, cu_t


def _oracle_row(qd_b, k_seq, v_seq, s, hk, grp, norm):
    """Oracle of row L-1 for the grp query heads of kv head hk: returns the
    result dicts of those heads (keys 0..grp-1)."""
    L, d = k_seq.shape[0], k_seq.shape[2]
    qs = np.zeros((1, L, grp, d), np.float16)
    qs[0, L - 1] = qd_b[hk * grp:(hk + 1) * grp]
    ks = k_seq[None, :, hk:hk + 1]
    vs = v_seq[None, :, hk:hk + 1]
    ss = None if s is None else s[hk:hk + 1]
    ref = oatt.attention_fwd(qs, ks, vs, ss, norm=norm, rows=[L - 1], want_p=True)
    return [ref[(0, j)] for j in range(grp)]


def _decode_and_compare(h, qd, k, v, cu, s, max_seqlen, norm="preorder", seqs=None, kv_heads=None):
    b_all = qd.shape[0]
    hq, hkv = qd.shape[1], k.shape[-2]
    grp = hq // hkv
    kc, km, vc, vm, cu_t = _build_cache(h, k, v, s, cu, max_seqlen)
    nm = h.NORM_PREORDER if norm == "preorder" else h.NORM_INCONSISTENT
    o, lse, pc, pm = h.hifa4_decode_fwd(to_gpu(qd), kc, km, vc, vm, None if s is None else to_gpu(s),
                                        cu_seqlens=cu_t, max_seqlen=max_seqlen, norm=nm, debug_p=True)
    o, lse, pc, pm = to_np(o), to_np(lse), to_np(pc), to_np(pm).view(np.uint32)
    worst = 0.0
    for b in (range(b_all) if seqs is None else seqs):
        if cu is None:
            k_seq, v_seq = k[b], v[b]
        else:
            k_seq, v_seq = k[cu[b]:cu[b + 1]], v[cu[b]:cu[b + 1]]
        L = k_seq.shape[0]
        if L == 0:
            continue                                # an empty sequence has no decode row
        nb = -(-L // 64)
        for hk in (range(hkv) if kv_heads is None else kv_heads):
            for j, r in enumerate(_oracle_row(qd[b], k_seq, v_seq, s, hk, grp, norm)):
                hh = hk * grp + j
                worst = max(worst, check_close(o[b, hh], r["o"][0], what=f"O seq {b} head {hh}"))
                check_close(lse[hh, b], r["lse"][0], atol=2e-3, rtol=0, what=f"LSE seq {b} head {hh}")
                assert np.array_equal(pc[hh, b, :nb], r["p_codes"][0, :nb]), (b, hh)
                assert np.array_equal(pm[hh, b, :nb], r["p_meta"][0, :nb]), (b, hh)
    return worst


def _last_queries(q, cu):
    return np.stack([q[cu[b + 1] - 1] for b in range(len(cu) - 1)])


@pytest.mark.parametrize("d,hq,hkv,lens,seed,smooth", [
    (128, 4, 1, (300, 65, 64, 1, 190), 1, True),     # GQA x4, ragged tails, single token
    (64, 2, 2, (129, 511), 2, False),                 # no GQA, D=64
    (256, 8, 1, (200, 33), 3, True),                  # GQA x8 (two rows per wave), D=256
    (128, 6, 2, (150, 700), 4, True),                 # GQA x3 (one wave idle)
    (128, 4, 1, (0, 300, 0, 65), 7, True),            # empty sequences (their rows are left untouched)
    (64, 24, 12, (100, 37), 8, True),                 # 12 kv heads: two workgroups per key range
    (128, 16, 2, (1000, 77), 14, True),               # GQA x8 at D=128
])
def test_decode_varlen_parity(h, d, hq, hkv, lens, seed, smooth):
    q, k, v, cu = small_case(heads_q=hq, heads_kv=hkv, head_dim=d, seqlens=lens, seed=seed)
    s = np.exp(np.random.default_rng(seed).uniform(-1, 1, (hkv, d))).astype(np.float32) if smooth else None
    qd = _last_queries(q, cu)
    for norm in ("preorder", "inconsistent"):
        _say("decode varlen", d, hq, hkv, lens, norm)
        _decode_and_compare(h, qd, k, v, cu, s, max(lens), norm=norm)


@pytest.mark.parametrize("d,hq,hkv,smooth", [(128, 8, 2, False), (128, 8, 2, True), (64, 6, 2, False),
                                             (256, 8, 1, True)])
def test_decode_query_edge_values(h, d, hq, hkv, smooth):
    """The score kernel quantizes the decode queries itself: every P^ code
    must still equal the oracle's for queries built from the quantizer's
    special cases."""
    lens = (300, 77)
    _, k, v, cu = small_case(heads_q=hq, heads_kv=hkv, head_dim=d, seqlens=lens, seed=21)
    s = np.exp(np.random.default_rng(21).uniform(-1, 1, (hkv, d))).astype(np.float32) if smooth else None
    qd = edge_rows(np.random.default_rng(22).standard_normal((len(lens), hq, d)).astype(np.float16), 22)
    _say("decode edge queries", d, hq, hkv, smooth)
    _decode_and_compare(h, qd, k, v, cu, s, max(lens))


def test_decode_fixed_length(h):
    """BSHD cache (every sequence max_seqlen tokens), three sequences."""
    q, k, v, cu = small_case(heads_q=4, heads_kv=2, head_dim=128, seqlens=(130, 130, 130), seed=9)
    qd = _last_queries(q, cu)
    k4 = k.reshape(3, 130, 2, 128)
    v4 = v.reshape(3, 130, 2, 128)
    _say("decode fixed length")
    _decode_and_compare(h, qd, k4, v4, None, None, 130)


@pytest.mark.parametrize("lens,d,hq,hkv,seed", [
    ((5000,), 128, 4, 1, 5),          # 79 blocks: score runs of 1, 40 splits of 2
    ((19000,), 128, 4, 1, 12),        # 297 blocks: 75 splits of 4
    ((33000,), 64, 2, 1, 6),          # 516 blocks: 65 splits of 8 (two 64-split passes of the merge)
    ((16384, 16384), 64, 16, 16, 13), # two workgroups of kv heads: score runs of 2, 64 splits of 4
])
def test_decode_many_splits(h, lens, d, hq, hkv, seed):
    """Long sequences, one shape per score-run and split length the launch
    picks from the block count, batch and kv heads."""
    q, k, v, cu = small_case(heads_q=hq, heads_kv=hkv, head_dim=d, seqlens=lens, seed=seed)
    s = np.exp(np.random.default_rng(seed).uniform(-1, 1, (hkv, d))).astype(np.float32)
    _say("decode long", lens, d, hq, hkv)
    _decode_and_compare(h, _last_queries(q, cu), k, v, cu, s, max(lens))


@pytest.mark.parametrize("lens,d,hq,hkv,seed,seqs,kv_heads", [
    # 64 kv heads in 8 workgroups, 58 blocks: runs and splits of 8, GQA x1
    ((3648, 3600, 3700, 3500, 3648, 3100, 3648, 3648), 64, 64, 64, 15, [0, 2, 5], [0, 37, 63]),
    # GQA x8 (two rows per softmax lane pass), 256 blocks in 2 workgroups of kv heads
    ((16384, 16000, 16384, 15000, 16384, 16300, 16384, 9000), 64, 128, 16, 16, [1, 7], [0, 9, 15]),
    # 64 blocks: runs and splits of 2, GQA x4, D=128
    ((4096, 4000, 4096, 3900, 4096, 4033, 4096, 2000), 128, 8, 2, 17, [0, 3, 7], [0, 1]),
])
def test_decode_fused_runs(h, lens, d, hq, hkv, seed, seqs, kv_heads):
    """Shapes whose splits fill the chip, so one kernel computes the scores
    of a split's blocks into LDS, publishes each row's run maximum and reads
    the earlier runs' maxima of its sequence: every P^ code of the sampled
    rows bit-exact."""
    _, k, v, cu = small_case(heads_q=hkv, heads_kv=hkv, head_dim=d, seqlens=lens, seed=seed)
    qd = np.random.default_rng(seed).standard_normal((len(lens), hq, d)).astype(np.float16)
    s = np.exp(np.random.default_rng(seed).uniform(-1, 1, (hkv, d))).astype(np.float32)
    _say("decode fused runs", len(lens), max(lens), d, hq, hkv)
    _decode_and_compare(h, qd, k, v, cu, s, max(lens), seqs=seqs, kv_heads=kv_heads)


def test_decode_cache_append(h):
    """The cache grows one token at a time: the K^ row of a new token
    quantized alone, and the V^ block holding it re-quantized from that
    block's fp16 tokens, equal the full-sequence quantization bit for bit;
    each step's decode matches the oracle."""
    import torch
    d, hq, hkv = 128, 4, 2
    q, k, v, cu = small_case(heads_q=hq, heads_kv=hkv, head_dim=d, seqlens=(131,), seed=11)
    s = np.exp(np.random.default_rng(11).uniform(-1, 1, (hkv, d))).astype(np.float32)
    s_t = to_gpu(s)
    cap = 192
    kc = torch.zeros((cap, hkv, d // 64, 32), dtype=torch.uint8, device="cuda")
    km = torch.zeros((cap, hkv, d // 64), dtype=torch.int32, device="cuda")
    vc = torch.zeros((1, cap // 64, hkv, d, 32), dtype=torch.uint8, device="cuda")
    vm = torch.zeros((1, cap // 64, hkv, d), dtype=torch.int32, device="cuda")
    k_t, v_t = to_gpu(k), to_gpu(v)
    for L in range(120, 132):
        if L == 120:
            _, _, kc0, km0 = h.hifa4_quantize_qk(None, k_t[:L].contiguous(), s_t,
                                                 cu_seqlens=to_gpu(np.array([0, L], np.int32)), max_seqlen=L)
            kc[:L], km[:L] = kc0, km0
        else:
            _, _, kc1, km1 = h.hifa4_quantize_qk(None, k_t[L - 1:L].contiguous(), s_t,
                                                 cu_seqlens=to_gpu(np.array([0, 1], np.int32)), max_seqlen=1)
            kc[L - 1], km[L - 1] = kc1[0], km1[0]
        j0 = (L - 1) // 64 * 64
        blocks = range(L // 64 + 1) if L == 120 else [j0 // 64]
        for J in blocks:
            t1 = min(L, 64 * J + 64)
            if t1 <= 64 * J:
                continue
            vb, vbm = h.hifa4_quantize_v(v_t[64 * J:t1].contiguous(),
                                         cu_seqlens=to_gpu(np.array([0, t1 - 64 * J], np.int32)),
                                         max_seqlen=t1 - 64 * J)
            vc[0, J], vm[0, J] = vb[0, 0], vbm[0, 0]
        nb = -(-L // 64)
        full = _build_cache(h, k[:L], v[:L], s, np.array([0, L], np.int32), L)
        assert torch.equal(kc[:L], full[0]) and torch.equal(km[:L], full[1])
        assert torch.equal(vc[:, :nb], full[2]) and torch.equal(vm[:, :nb], full[3])
        qd = q[L - 1][None]
        cu_t = to_gpu(np.array([0, L], np.int32))
        o, lse, pc, pm = h.hifa4_decode_fwd(to_gpu(qd), kc[:L], km[:L], vc[:, :nb].contiguous(),
                                            vm[:, :nb].contiguous(), s_t, cu_seqlens=cu_t, max_seqlen=L,
                                            debug_p=True)
        o, lse, pc, pm = to_np(o), to_np(lse), to_np(pc), to_np(pm).view(np.uint32)
        for hk in range(hkv):
            for j, r in enumerate(_oracle_row(qd[0], k[:L], v[:L], s, hk, hq // hkv, "preorder")):
                hh = hk * (hq // hkv) + j
                check_close(o[0, hh], r["o"][0], what=f"O step {L} head {hh}")
                check_close(lse[hh, 0], r["lse"][0], atol=2e-3, rtol=0, what="LSE")
                assert np.array_equal(pc[hh, 0, :nb], r["p_codes"][0, :nb]), (L, hh)
                assert np.array_equal(pm[hh, 0, :nb], r["p_meta"][0, :nb]), (L, hh)
    _say("decode append ok")


def test_decode_b8_l32768_sampled(h):
    """The decode workload at full size in the benchmark's launch shape (8
    sequences of 32768 cached tokens, Qwen3-8B heads, Smooth-QK scales from
    the Qwen3-shaped calibration draw): sampled sequences and kv heads, every
    P^ code of those rows bit-exact, O and LSE."""
    w = WORKLOADS["decode_b8_l32768"]
    qd, k, v, _ = make_decode_inputs(w)
    qc, kc = make_calibration(WORKLOADS[w.calib_from], n=4)
    s, _ = osmooth.calibrate(qc, kc, w.heads_kv, w.alpha)
    _say("decode_b8_l32768 sampled")
    _decode_and_compare(h, qd, k, v, None, s, w.seqlen, seqs=[0, 7], kv_heads=[0, 5])


def test_decode_graph_replay(h):
    """The decode step captured as a HIP graph: every replay, with eager work
    and synchronizations between replays, equals the eager call bit for bit
    (the library's launches record no memsets)."""
    import torch
    q, k, v, cu = small_case(heads_q=4, heads_kv=2, head_dim=128, seqlens=(700, 65), seed=13)
    s = np.exp(np.random.default_rng(13).uniform(-1, 1, (2, 128))).astype(np.float32)
    kc, km, vc, vm, cu_t = _build_cache(h, k, v, s, cu, 700)
    qd, s_t = to_gpu(_last_queries(q, cu)), to_gpu(s)
    ws = h.Workspace()
    o_ref, l_ref = h.hifa4_decode_fwd(qd, kc, km, vc, vm, s_t, cu_seqlens=cu_t, max_seqlen=700, workspace=ws)
    o_ref, l_ref = o_ref.clone(), l_ref.clone()
    out = torch.empty_like(o_ref)
    lse = torch.empty_like(l_ref)
    kw = dict(cu_seqlens=cu_t, max_seqlen=700, workspace=ws, out=out, lse=lse)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        h.hifa4_decode_fwd(qd, kc, km, vc, vm, s_t, **kw)
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        h.hifa4_decode_fwd(qd, kc, km, vc, vm, s_t, **kw)
    for i in range(4):
        out.zero_()
        lse.zero_()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, o_ref), i
        assert torch.equal(lse, l_ref), i
        h.hifa4_decode_fwd(qd, kc, km, vc, vm, s_t, cu_seqlens=cu_t, max_seqlen=700)   # eager work between
        torch.cuda.synchronize()
    _say("decode graph replays ok")


def _fused_case():
    """8 sequences of about 4096 tokens, 2 kv heads, GQA x4, D=128: 64 blocks
    per row in splits of 2, 256 split workgroups, so scores and splits run in
    one kernel that waits on run maxima."""
    lens = (4096, 4000, 4096, 3900, 4096, 4033, 4096, 2000)
    _, k, v, cu = small_case(heads_q=2, heads_kv=2, head_dim=128, seqlens=lens, seed=31)
    s = np.exp(np.random.default_rng(31).uniform(-1, 1, (2, 128))).astype(np.float32)
    return lens, k, v, cu, s


def test_decode_graph_replay_fused(h):
    """The fused decode step captured once and replayed back to back with a
    new query written in place before each replay (no eager decode call in
    between): every replay equals an eager call on the same query bit for
    bit, and its P^ codes equal the oracle's on sampled rows.  A replay reuses
    the captured call's tag, so this fails if a split can take the previous
    replay's run maxima for its own."""
    import torch
    lens, k, v, cu, s = _fused_case()
    hq, hkv, d = 8, 2, 128
    kc, km, vc, vm, cu_t = _build_cache(h, k, v, s, cu, max(lens))
    s_t = to_gpu(s)
    rng = np.random.default_rng(32)
    queries = [(rng.standard_normal((len(lens), hq, d)) * (1.0 + 2.0 * i)).astype(np.float16) for i in range(3)]
    q_buf = to_gpu(queries[0])
    ws = h.Workspace()
    kw = dict(cu_seqlens=cu_t, max_seqlen=max(lens), workspace=ws, debug_p=True)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        h.hifa4_decode_fwd(q_buf, kc, km, vc, vm, s_t, **kw)
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        g_o, g_l, g_pc, g_pm = h.hifa4_decode_fwd(q_buf, kc, km, vc, vm, s_t, **kw)
    got = []
    for qi in queries:
        q_buf.copy_(to_gpu(qi))
        graph.replay()
        got.append((g_o.clone(), g_l.clone(), g_pc.clone(), g_pm.clone()))
    torch.cuda.synchronize()
    for i, qi in enumerate(queries):
        _say("fused replay", i)
        o, l, pc, pm = h.hifa4_decode_fwd(to_gpu(qi), kc, km, vc, vm, s_t, cu_seqlens=cu_t,
                                          max_seqlen=max(lens), debug_p=True)
        torch.cuda.synchronize()
        assert torch.equal(got[i][0], o) and torch.equal(got[i][1], l), f"replay {i} differs from eager"
        assert torch.equal(got[i][2], pc) and torch.equal(got[i][3], pm), f"replay {i} P^ differs from eager"
        pc_n, pm_n = to_np(got[i][2]), to_np(got[i][3]).view(np.uint32)
        for b in (0, 5):
            k_seq, v_seq = k[cu[b]:cu[b + 1]], v[cu[b]:cu[b + 1]]
            nb = -(-k_seq.shape[0] // 64)
            for hk in range(hkv):
                for j, r in enumerate(_oracle_row(qi[b], k_seq, v_seq, s, hk, hq // hkv, "preorder")):
                    hh = hk * (hq // hkv) + j
                    assert np.array_equal(pc_n[hh, b, :nb], r["p_codes"][0, :nb]), (i, b, hh)
                    assert np.array_equal(pm_n[hh, b, :nb], r["p_meta"][0, :nb]), (i, b, hh)
    _say("fused graph replays ok")


def test_decode_wait_gives_up(h):
    """The bounded wait of the fused kernel made to give up from the host (no
    run maxima published, 16 polls per wait): every kernel ends and each row,
    whose later splits all lost their wait, comes out NaN rather than
    silently wrong; the next normal call is correct again."""
    import torch
    lens, k, v, cu, s = _fused_case()
    hq, d = 8, 128
    kc, km, vc, vm, cu_t = _build_cache(h, k, v, s, cu, max(lens))
    qd = np.random.default_rng(33).standard_normal((len(lens), hq, d)).astype(np.float16)
    o, l = h.hifa4_decode_fwd(to_gpu(qd), kc, km, vc, vm, to_gpu(s), cu_seqlens=cu_t, max_seqlen=max(lens),
                              test_no_publish=True)
    torch.cuda.synchronize()
    assert torch.isnan(o).all() and torch.isnan(l).all(), "a wait that gave up must poison its row"
    _say("decode give-up rows are NaN")
    _decode_and_compare(h, qd, k, v, cu, s, max(lens), seqs=[1, 7], kv_heads=[0, 1])


@pytest.mark.parametrize("kind,jump_block,lens", [
    ("wipe", 2, (450, 200)),          # the jump opens the second split: the merge wipes the first
    ("wipe", 1, (450, 200)),          # the jump inside the first split
    ("renorm", 0, (450, 400)),
    ("wipe", 2, (4096,) * 8),         # fused shape (256 split workgroups)
    ("renorm", 0, (4096,) * 8),
])
def test_decode_running_max_special_paths(h, kind, jump_block, lens):
    """The decode row (L-1) of inputs whose running maximum jumps by more
    than 25 log2 units (a rescale factor of 0, so earlier blocks or splits
    are wiped) or rises over 64 units in smaller steps: every P^ code of the
    sampled rows bit-exact, O and LSE, both normalizers."""
    from _jump import check_jumps, jump_case
    d, hq, hkv = 128, 4, 1
    q, k, v, cu = jump_case(kind, lens, hq, hkv, d, seed=81, jump_block=jump_block)
    check_jumps(kind, q, k, cu, d, "hif4", last_row_only=True, min_hits=len(lens))
    qd = _last_queries(q, cu)
    seqs = None if len(lens) <= 2 else [0, 5]
    for norm in ("preorder", "inconsistent"):
        _say("decode running max", kind, jump_block, len(lens), norm)
        _decode_and_compare(h, qd, k, v, cu, None, max(lens), norm=norm, seqs=seqs)
