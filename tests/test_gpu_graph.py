"""The prefill forward captured as a HIP graph (the library launches two
kernels per call and records no memsets, so a call captures as it is):
replayed back to back with new Q, K and V written in place before each
replay, with eager calls and synchronizations between the replays, every
replay equals an eager call on the same inputs bit for bit, and its O and
LSE are within the parity bar of the oracle on sampled rows.  The same for
the entry point without allocation, whose workspace is the library's static
scratch array (the capture records its address)."""
import sys

import numpy as np
import pytest

from oracle import attention as oatt
from paper_2607_04302_amd.workloads import small_case

from _gpu_util import LSE_ATOL, check_close, to_gpu, to_np

pytestmark = pytest.mark.gpu

LENS = (300, 77, 129)
HQ, HKV, D = 4, 2, 128


@pytest.fixture(scope="module")
def h():
    import paper_2607_04302_amd as mod
    mod.load_library()
    return mod


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _inputs(seed):
    q, k, v, cu = small_case(heads_q=HQ, heads_kv=HKV, head_dim=D, seqlens=LENS, seed=seed)
    s = np.exp(np.random.default_rng(seed).uniform(-1, 1, (HKV, D))).astype(np.float32)
    return q, k, v, cu, s


def _replay_and_check(h, call, name):
    import torch
    sets = [_inputs(70 + i) for i in range(3)]
    cu = sets[0][3]
    assert all(np.array_equal(x[3], cu) for x in sets)
    q_buf, k_buf, v_buf, s_buf = (to_gpu(x) for x in (sets[0][0], sets[0][1], sets[0][2], sets[0][4]))
    cu_t = to_gpu(cu)
    out = torch.empty_like(q_buf)
    lse = torch.empty((HQ, q_buf.shape[0]), dtype=torch.float32, device=q_buf.device)
    kw = dict(cu_seqlens=cu_t, max_seqlen=max(LENS), out=out, lse=lse)
    # warm-up on a side stream (sizes any workspace before the capture)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call(q_buf, k_buf, v_buf, s_buf, **kw)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call(q_buf, k_buf, v_buf, s_buf, **kw)
    torch.cuda.synchronize()
    for i, (q, k, v, _, s) in enumerate(sets):
        _say(name, "replay", i)
        q_buf.copy_(to_gpu(q))
        k_buf.copy_(to_gpu(k))
        v_buf.copy_(to_gpu(v))
        s_buf.copy_(to_gpu(s))
        out.zero_()
        lse.zero_()
        graph.replay()
        torch.cuda.synchronize()
        o_g, l_g = out.clone(), lse.clone()
        # eager work between replays: the same inputs through fresh buffers
        o_e, l_e = call(to_gpu(q), to_gpu(k), to_gpu(v), to_gpu(s), cu_seqlens=cu_t, max_seqlen=max(LENS))
        torch.cuda.synchronize()
        assert torch.equal(o_g, o_e) and torch.equal(l_g, l_e), f"{name}: replay {i} differs from the eager call"
        ref = oatt.attention_fwd(q, k, v, s, cu_seqlens=cu, heads=[0, HQ - 1], rows=[0, 63, 64, 76, 128, 299])
        o_n, l_n = to_np(o_g), to_np(l_g)
        for (b, hh), r in ref.items():
            tok = cu[b] + r["rows"]
            check_close(o_n[tok, hh], r["o"], what=f"{name} replay {i} O seq {b} head {hh}")
            check_close(l_n[hh, tok], r["lse"], atol=LSE_ATOL, rtol=0.0, what=f"{name} replay {i} LSE")
    del graph


def test_prefill_graph_replay(h):
    ws = h.Workspace()

    def call(q, k, v, s, **kw):
        return h.hifa4_attention_fwd(q, k, v, s, workspace=ws, **kw)

    _replay_and_check(h, call, "prefill")


def test_prefill_noalloc_graph_replay(h):
    _replay_and_check(h, h.hifa4_attention_fwd_noalloc, "no-alloc prefill")
