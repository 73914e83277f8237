"""C ABI: the library loads, exports every entry point of include/hifa4.h, and
rejects invalid arguments with status codes before any GPU work."""
import ctypes
import os
import re

import pytest

import paper_2607_04302_amd as h

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "hifa4.h")).read()
    return sorted(set(re.findall(r"\b(hifa4_[a-z0-9_]+)\s*\(", text)))


def test_header_and_binding_agree():
    assert set(_declared()) == set(h.EXPORTED)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(h.LIB_PATH):
        pytest.skip("libhifa4.so not built")
    return h.load_library()


def test_exports(lib):
    for name in _declared():
        assert hasattr(lib, name), name


def _p(**kw):
    base = dict(batch=1, num_heads_q=4, num_heads_kv=2, head_dim=128, max_seqlen=128,
                cu_seqlens=None, total_tokens=0, causal=1)
    base.update(kw)
    return h.Problem(**base)


FAKE = 1 << 12          # an aligned non-NULL address; never dereferenced (validation fails first)


def _fwd(lib, p, opt=None, ptr=FAKE, ws=1 << 30):
    opt = opt or h.FwdOptions(0, 0, 0, None, None, None)
    return lib.hifa4_attention_fwd(ctypes.byref(p), ctypes.byref(opt), ptr, ptr, ptr, None, ptr, ptr,
                                   ptr, ws, None)


def test_validation_codes(lib):
    assert _fwd(lib, _p(head_dim=96)) == -2
    assert "head_dim" in h.hifa4_last_error()
    assert _fwd(lib, _p(num_heads_q=3, num_heads_kv=2)) == -2
    assert _fwd(lib, _p(causal=0)) == -2
    assert _fwd(lib, _p(batch=0)) == -1
    assert _fwd(lib, _p(), ptr=None) == -1
    assert _fwd(lib, _p(), opt=h.FwdOptions(7, 0, 0, None, None, None)) == -1
    assert _fwd(lib, _p(), opt=h.FwdOptions(0, 0, 1, None, None, None)) == -1      # smooth without s
    assert _fwd(lib, _p(), opt=h.FwdOptions(0, 0, 0, FAKE, None, None)) == -1      # half a debug dump
    assert _fwd(lib, _p(), opt=h.FwdOptions(0, 1, 0, None, None, None, 1)) == -2   # Q-Mean with fp16 operands
    assert "q_mean" in h.hifa4_last_error()
    assert _fwd(lib, _p(), ws=16) == -3
    assert "workspace" in h.hifa4_last_error()
    # P^ dump windows: outside the problem, negative, or a begin without a count
    tokens = _p().batch * _p().max_seqlen
    for win in ((0, _p().num_heads_q + 1, 0, 0), (1, _p().num_heads_q, 0, 0), (0, 0, 0, tokens + 1),
                (-1, 1, 0, 0), (0, 0, 5, 0), (0, 0, tokens - 1, 2), (0, -1, 0, 0)):
        assert _fwd(lib, _p(), opt=h.FwdOptions(0, 0, 0, FAKE, FAKE, None, 0, 0, *win)) == -1, win
        assert "debug window" in h.hifa4_last_error()
    assert lib.hifa4_selftest_exp2(None, None, -1, None) == -1


def test_noalloc_refuses_oversized_before_any_work(lib):
    """The no-allocation entry point checks the workspace a problem needs
    against its static array before it touches the GPU (this runs without
    one)."""
    p = _p(max_seqlen=16384, num_heads_q=32, num_heads_kv=8)
    opt = h.FwdOptions(0, 0, 0, None, None, None)
    assert lib.hifa4_workspace_bytes(ctypes.byref(p), ctypes.byref(opt)) > h.NOALLOC_SCRATCH_BYTES
    assert lib.hifa4_attention_fwd_noalloc(ctypes.byref(p), ctypes.byref(opt), FAKE, FAKE, FAKE, None, FAKE,
                                           FAKE, None) == -3
    assert "at most" in h.hifa4_last_error()
    assert lib.hifa4_attention_fwd_noalloc(ctypes.byref(_p(head_dim=96)), ctypes.byref(opt), FAKE, FAKE, FAKE,
                                           None, FAKE, FAKE, None) == -2


def test_workspace_sizes(lib):
    p = _p(max_seqlen=4096, num_heads_q=32, num_heads_kv=8)
    o = h.FwdOptions(0, 0, 0, None, None, None)
    n = lib.hifa4_workspace_bytes(ctypes.byref(p), ctypes.byref(o))
    # 64 blocks x 8 kv heads x (K: 2 key halves x 2 groups x 2 operands of
    # 1536 B + 512 B of scale words; V: 4 channel tiles x 2 operands of 1536 B
    # + 512 B of scale words)
    assert n == 64 * 8 * 25600
    # Q-Mean adds 256 B of key sums per chunk, rounded to a whole KiB
    oq = h.FwdOptions(0, 0, 0, None, None, None, 1)
    assert lib.hifa4_workspace_bytes(ctypes.byref(p), ctypes.byref(oq)) == 64 * 8 * 26624
    o16 = h.FwdOptions(0, 1, 0, None, None, None)
    assert lib.hifa4_workspace_bytes(ctypes.byref(p), ctypes.byref(o16)) == 64 * 8 * 32768
    assert lib.hifa4_workspace_bytes(ctypes.byref(_p(head_dim=80)), ctypes.byref(o)) == 0


def _dec(lib, p, opt=None, ptr=FAKE, ws=1 << 30):
    opt = opt or h.FwdOptions(0, 0, 0, None, None, None)
    return lib.hifa4_decode_fwd(ctypes.byref(p), ctypes.byref(opt), ptr, ptr, ptr, ptr, ptr, None, ptr, ptr,
                                ptr, ws, None)


def test_decode_validation_codes(lib):
    assert _dec(lib, _p(head_dim=96)) == -2
    assert _dec(lib, _p(), opt=h.FwdOptions(0, 1, 0, None, None, None)) == -2     # fp16 operands
    assert "HIF4" in h.hifa4_last_error()
    assert _dec(lib, _p(), opt=h.FwdOptions(0, 0, 0, None, None, None, 1)) == -2  # Q-Mean
    assert "q_mean" in h.hifa4_last_error()
    assert _dec(lib, _p(num_heads_q=64, num_heads_kv=2)) == -2                   # GQA group of 32
    assert _dec(lib, _p(num_heads_q=32, num_heads_kv=2)) == -2                   # GQA group of 16
    assert "at most 8" in h.hifa4_last_error()
    assert _dec(lib, _p(), ptr=None) == -1
    assert _dec(lib, _p(), opt=h.FwdOptions(0, 0, 1, None, None, None)) == -1     # smooth without s
    assert _dec(lib, _p(), opt=h.FwdOptions(0, 0, 0, None, FAKE, None)) == -1     # half a debug dump
    assert _dec(lib, _p(), opt=h.FwdOptions(3, 0, 0, None, None, None)) == -1
    assert _dec(lib, _p(), ws=16) == -3


def test_decode_workspace_sizes(lib):
    # B=2, Hq=32, D=128, S=4096: scores 2*32*64*64*2 B, block maxima 2*32*64*2 B, and
    # per row and split partial O (128 fp32) and (l, factor product, max).
    # Splits of 8 or 4 blocks would leave 16 or 32 workgroups: this shape takes
    # the shortest splits, 2 blocks (32 per row).
    p = _p(batch=2, max_seqlen=4096, num_heads_q=32, num_heads_kv=8)
    rows = 2 * 32
    want = rows * 64 * 64 * 2 + rows * 64 * 2 + rows * 32 * 128 * 4 + rows * 32 * 16
    assert lib.hifa4_decode_workspace_bytes(ctypes.byref(p)) == want
    # 8 sequences of 4096 tokens: splits of 2 blocks fill 256 workgroups, so
    # one kernel takes scores and splits (run maxima instead of scores)
    p = _p(batch=8, max_seqlen=4096, num_heads_q=32, num_heads_kv=8)
    rows = 8 * 32
    want = rows * 32 * 128 * 4 + rows * 32 * 16 + rows * 32 * 8
    assert lib.hifa4_decode_workspace_bytes(ctypes.byref(p)) == want
    # 100 tokens (2 blocks) pad the block maxima of a row to 8 entries
    p = _p(batch=3, max_seqlen=100, num_heads_q=4, num_heads_kv=1)
    rows = 3 * 4
    want = 256 * ((rows * 2 * 64 * 2 + 255) // 256) + 256 + 256 * ((rows * 1 * 128 * 4 + 255) // 256) + 256
    assert lib.hifa4_decode_workspace_bytes(ctypes.byref(p)) == want
    # 8 sequences of 32768 tokens: runs and splits of 8 blocks (512
    # workgroups), one kernel for both, so no scores or block maxima, but an
    # 8-byte run maximum per row and run
    p = _p(batch=8, max_seqlen=32768, num_heads_q=32, num_heads_kv=8)
    rows = 8 * 32
    want = rows * 64 * 128 * 4 + rows * 64 * 16 + rows * 64 * 8
    assert lib.hifa4_decode_workspace_bytes(ctypes.byref(p)) == want
    assert lib.hifa4_decode_workspace_bytes(ctypes.byref(_p(head_dim=80))) == 0


def test_alignment_is_checked(lib):
    """fp16 tensors, scales, code buffers, workspace and P^ dumps need 16-byte
    alignment, metadata and LSE 4 bytes; violations fail before any launch."""
    p = _p()
    for bad in (FAKE + 2, FAKE + 8):
        assert lib.hifa4_attention_fwd(ctypes.byref(p), ctypes.byref(h.FwdOptions(0, 0, 0, None, None, None)),
                                       bad, FAKE, FAKE, None, FAKE, FAKE, FAKE, 1 << 30, None) == -1
        assert "aligned" in h.hifa4_last_error()
        assert lib.hifa4_attention_fwd(ctypes.byref(p), ctypes.byref(h.FwdOptions(0, 0, 0, None, None, None)),
                                       FAKE, FAKE, FAKE, None, FAKE, FAKE, bad, 1 << 30, None) == -1    # workspace
        assert lib.hifa4_decode_fwd(ctypes.byref(p), ctypes.byref(h.FwdOptions(0, 0, 0, None, None, None)),
                                    FAKE, bad, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, 1 << 30, None) == -1
        assert lib.hifa4_quantize_qk(ctypes.byref(p), FAKE, FAKE, None, FAKE, FAKE, bad, FAKE, None) == -1
        assert lib.hifa4_quantize_v(ctypes.byref(p), FAKE, bad, FAKE, None) == -1
    assert lib.hifa4_attention_fwd(ctypes.byref(p), ctypes.byref(h.FwdOptions(0, 0, 0, None, None, None)),
                                   FAKE, FAKE, FAKE, None, FAKE, FAKE + 2, FAKE, 1 << 30, None) == -1    # LSE
    assert lib.hifa4_quantize_v(ctypes.byref(p), FAKE, FAKE, FAKE + 2, None) == -1                    # meta
    assert lib.hifa4_decode_fwd(ctypes.byref(p), ctypes.byref(h.FwdOptions(0, 0, 0, None, None, None)),
                                FAKE, FAKE, FAKE + 1, FAKE, FAKE, None, FAKE, FAKE, FAKE, 1 << 30, None) == -1
