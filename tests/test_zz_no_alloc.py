"""The entry point that allocates nothing (hifa4_attention_fwd_noalloc, for
callers that cannot allocate device memory), through the C ABI: two calls in
a row on one GPU, the second on a smaller problem, each equal bit for bit to
hifa4_attention_fwd with a caller workspace on the same inputs, O and LSE
within the parity bar of the oracle on sampled rows; a problem larger than
the static scratch array is refused before any work is enqueued."""
import numpy as np
import pytest

from oracle import attention as oatt
from paper_2607_04302_amd.workloads import small_case

from _gpu_util import check_close, to_gpu, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def h():
    import paper_2607_04302_amd as mod
    mod.load_library()
    return mod


def _case(h, lens, hq, hkv, d, seed, rows):
    import torch
    q, k, v, cu = small_case(heads_q=hq, heads_kv=hkv, head_dim=d, seqlens=lens, seed=seed)
    s = np.exp(np.random.default_rng(seed).uniform(-1, 1, (hkv, d))).astype(np.float32)
    args = (to_gpu(q), to_gpu(k), to_gpu(v), to_gpu(s))
    kw = dict(cu_seqlens=to_gpu(cu), max_seqlen=max(lens))
    o_n, l_n = h.hifa4_attention_fwd_noalloc(*args, **kw)
    torch.cuda.synchronize()
    o_w, l_w = h.hifa4_attention_fwd(*args, workspace=h.Workspace(), **kw)
    torch.cuda.synchronize()
    assert torch.equal(o_n, o_w) and torch.equal(l_n, l_w), "no-alloc result differs from the workspace call"
    ref = oatt.attention_fwd(q, k, v, s, cu_seqlens=cu, heads=[0, hq - 1], rows=rows)
    o_n, l_n = to_np(o_n), to_np(l_n)
    for (b, hh), r in ref.items():
        tok = cu[b] + r["rows"]
        check_close(o_n[tok, hh], r["o"], what=f"no-alloc O seq {b} head {hh}")
        check_close(l_n[hh, tok], r["lse"], atol=2e-3, rtol=0, what="no-alloc LSE")


def test_noalloc_two_calls_second_smaller(h):
    # 8 kv heads, D=128, 4096 tokens: 13.1 MB of the 32 MiB array
    _case(h, (4096,), 32, 8, 128, 91, rows=[0, 63, 64, 2047, 4095])
    # then a smaller ragged problem on the same array (stale contents of the
    # first call stay beyond what this one writes)
    _case(h, (300, 77), 4, 2, 64, 92, rows=[0, 1, 64, 76, 299])


def test_noalloc_refuses_oversized(h):
    import torch
    q = torch.zeros((1, 16384, 32, 128), dtype=torch.float16, device="cuda")
    k = torch.zeros((1, 16384, 8, 128), dtype=torch.float16, device="cuda")
    with pytest.raises(h.Hifa4Error, match="at most"):
        h.hifa4_attention_fwd_noalloc(q, k, k)
