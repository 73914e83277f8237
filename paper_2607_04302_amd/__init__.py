"""HiFA4 on MI355X: Python binding of libhifa4 (the C ABI in include/hifa4.h).

The binding only marshals arguments: torch tensors supply device memory and
the current HIP stream; every step of the computation runs in the library's
HIP kernels.  The shared library is loaded on first use from this package's
directory and a missing or stale build raises immediately -- there is no
fallback implementation.

Names mirror the C entry points:
  hifa4_calibrate_smooth_qk, hifa4_calibrate_smooth_qk_layers, hifa4_quantize_qk, hifa4_quantize_v,
  hifa4_attention_fwd, hifa4_workspace_bytes, hifa4_decode_fwd,
  hifa4_decode_workspace_bytes, hifa4_selftest_exp2, hifa4_last_error.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libhifa4.so")

NORM_PREORDER, NORM_INCONSISTENT = 0, 1
OPERANDS_HIF4, OPERANDS_FP16, OPERANDS_P_ONLY = 0, 1, 2
STATUS = {0: "HIFA4_OK", -1: "HIFA4_ERR_INVALID_ARGUMENT", -2: "HIFA4_ERR_UNSUPPORTED",
          -3: "HIFA4_ERR_WORKSPACE", -4: "HIFA4_ERR_HIP"}

EXPORTED = ("hifa4_workspace_bytes", "hifa4_calibrate_workspace_bytes", "hifa4_calibrate_smooth_qk",
            "hifa4_calibrate_smooth_qk_layers",
            "hifa4_quantize_qk", "hifa4_quantize_v", "hifa4_attention_fwd", "hifa4_decode_workspace_bytes",
            "hifa4_decode_fwd", "hifa4_selftest_exp2", "hifa4_last_error", "hifa4_attention_fwd_noalloc")
NOALLOC_SCRATCH_BYTES = 32 << 20


class Problem(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_heads_q", ctypes.c_int32),
                ("num_heads_kv", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("max_seqlen", ctypes.c_int32), ("cu_seqlens", ctypes.c_void_p),
                ("total_tokens", ctypes.c_int32), ("causal", ctypes.c_int32)]


class FwdOptions(ctypes.Structure):
    _fields_ = [("norm", ctypes.c_int32), ("operands", ctypes.c_int32), ("smooth_qk", ctypes.c_int32),
                ("debug_p_codes", ctypes.c_void_p), ("debug_p_meta", ctypes.c_void_p),
                ("timing_events", ctypes.c_void_p), ("q_mean", ctypes.c_int32),
                ("test_decode_no_publish", ctypes.c_int32),
                ("debug_head_begin", ctypes.c_int32), ("debug_head_count", ctypes.c_int32),
                ("debug_token_begin", ctypes.c_int32), ("debug_token_count", ctypes.c_int32)]


class CalibReport(ctypes.Structure):
    _fields_ = [("rho_k", ctypes.c_double), ("t_kq", ctypes.c_double), ("branch", ctypes.c_int32),
                ("alpha_used", ctypes.c_float)]


class Hifa4Error(RuntimeError):
    pass


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libhifa4.so (once).  Raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"libhifa4.so not found at {path}; build it first "
                          "(python -m paper_2607_04302_amd.build or __graft_entry__.build())")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    vp, sz = ctypes.c_void_p, ctypes.c_size_t
    lib.hifa4_workspace_bytes.restype = sz
    lib.hifa4_workspace_bytes.argtypes = [P(Problem), P(FwdOptions)]
    lib.hifa4_calibrate_workspace_bytes.restype = sz
    lib.hifa4_calibrate_workspace_bytes.argtypes = [P(Problem), ctypes.c_int32]
    lib.hifa4_calibrate_smooth_qk.restype = ctypes.c_int
    lib.hifa4_calibrate_smooth_qk.argtypes = [P(Problem), ctypes.c_int32, vp, vp, ctypes.c_float, vp,
                                              P(CalibReport), vp, sz, vp]
    lib.hifa4_calibrate_smooth_qk_layers.restype = ctypes.c_int
    lib.hifa4_calibrate_smooth_qk_layers.argtypes = [P(Problem), ctypes.c_int32, ctypes.c_int32, vp, vp,
                                                     ctypes.c_float, vp, P(CalibReport), vp, sz, vp]
    lib.hifa4_quantize_qk.restype = ctypes.c_int
    lib.hifa4_quantize_qk.argtypes = [P(Problem), vp, vp, vp, vp, vp, vp, vp, vp]
    lib.hifa4_quantize_v.restype = ctypes.c_int
    lib.hifa4_quantize_v.argtypes = [P(Problem), vp, vp, vp, vp]
    lib.hifa4_attention_fwd.restype = ctypes.c_int
    lib.hifa4_attention_fwd.argtypes = [P(Problem), P(FwdOptions), vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.hifa4_attention_fwd_noalloc.restype = ctypes.c_int
    lib.hifa4_attention_fwd_noalloc.argtypes = [P(Problem), P(FwdOptions), vp, vp, vp, vp, vp, vp, vp]
    lib.hifa4_decode_workspace_bytes.restype = sz
    lib.hifa4_decode_workspace_bytes.argtypes = [P(Problem)]
    lib.hifa4_decode_fwd.restype = ctypes.c_int
    lib.hifa4_decode_fwd.argtypes = [P(Problem), P(FwdOptions), vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.hifa4_selftest_exp2.restype = ctypes.c_int
    lib.hifa4_selftest_exp2.argtypes = [vp, vp, ctypes.c_int64, vp]
    lib.hifa4_last_error.restype = ctypes.c_char_p
    lib.hifa4_last_error.argtypes = []
    _lib = lib
    return lib


def hifa4_last_error() -> str:
    return load_library().hifa4_last_error().decode()


def _check(status: int, what: str):
    if status != 0:
        raise Hifa4Error(f"{what}: {STATUS.get(status, status)}: {hifa4_last_error()}")


def _torch():
    import torch
    return torch


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(device=None) -> int:
    torch = _torch()
    return torch.cuda.current_stream(device).cuda_stream


def _require(t, dtype, name):
    torch = _torch()
    if t is None:
        return
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    del torch


@dataclass
class Shape:
    batch: int
    heads_q: int
    heads_kv: int
    head_dim: int
    max_seqlen: int
    tokens: int
    cu_seqlens: object = None

    def problem(self) -> Problem:
        return Problem(self.batch, self.heads_q, self.heads_kv, self.head_dim, self.max_seqlen,
                       _ptr(self.cu_seqlens), self.tokens if self.cu_seqlens is not None else 0, 1)


def shape_of(q, k, cu_seqlens=None, max_seqlen=None) -> Shape:
    """Problem shape from Q [B,S,Hq,D] (BSHD) or Q [T,Hq,D] + cu_seqlens (THD)."""
    if cu_seqlens is None:
        if q.dim() != 4:
            raise ValueError("fixed-length inputs are [batch, seqlen, heads, dim]")
        b, s, hq, d = q.shape
        return Shape(b, hq, k.shape[2], d, s, b * s)
    if q.dim() != 3:
        raise ValueError("variable-length inputs are [total_tokens, heads, dim] with cu_seqlens")
    if max_seqlen is None:
        raise ValueError("max_seqlen is required with cu_seqlens")
    _require(cu_seqlens, _torch().int32, "cu_seqlens")
    t, hq, d = q.shape
    return Shape(cu_seqlens.numel() - 1, hq, k.shape[1], d, int(max_seqlen), t, cu_seqlens)


def hifa4_workspace_bytes(shape: Shape, operands: int = OPERANDS_HIF4, q_mean: bool = False) -> int:
    lib = load_library()
    p = shape.problem()
    o = FwdOptions(NORM_PREORDER, operands, 0, None, None, None, 1 if q_mean else 0)
    return int(lib.hifa4_workspace_bytes(ctypes.byref(p), ctypes.byref(o)))


def hifa4_calibrate_smooth_qk(q_cal, k_cal, alpha: float):
    """q_cal [n, S, Hq, D], k_cal [n, S, Hkv, D] fp16 on the GPU.  Returns
    (s fp32 [Hkv, D] on the GPU, report dict).  Synchronizes the stream."""
    torch = _torch()
    _require(q_cal, torch.float16, "q_cal")
    _require(k_cal, torch.float16, "k_cal")
    lib = load_library()
    n, s, hq, d = q_cal.shape
    hkv = k_cal.shape[2]
    p = Problem(1, hq, hkv, d, s, None, 0, 1)
    ws_bytes = int(lib.hifa4_calibrate_workspace_bytes(ctypes.byref(p), n))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=q_cal.device)
    out = torch.empty((hkv, d), dtype=torch.float32, device=q_cal.device)
    rep = CalibReport()
    _check(lib.hifa4_calibrate_smooth_qk(ctypes.byref(p), n, _ptr(q_cal), _ptr(k_cal), float(alpha),
                                         _ptr(out), ctypes.byref(rep), _ptr(ws), ws_bytes,
                                         _stream(q_cal.device)), "hifa4_calibrate_smooth_qk")
    return out, {"rho_k": rep.rho_k, "t_kq": rep.t_kq, "branch": rep.branch, "alpha_used": rep.alpha_used}


def hifa4_calibrate_smooth_qk_layers(q_cal, k_cal, alpha: float):
    """q_cal [L, n, S, Hq, D], k_cal [L, n, S, Hkv, D] fp16 on the GPU (L
    layers).  Returns (s fp32 [L, Hkv, D] on the GPU, list of L report dicts).
    Synchronizes the stream."""
    torch = _torch()
    _require(q_cal, torch.float16, "q_cal")
    _require(k_cal, torch.float16, "k_cal")
    lib = load_library()
    n_layers, n, s, hq, d = q_cal.shape
    hkv = k_cal.shape[3]
    p = Problem(1, hq, hkv, d, s, None, 0, 1)
    ws_bytes = int(lib.hifa4_calibrate_workspace_bytes(ctypes.byref(p), n))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=q_cal.device)
    out = torch.empty((n_layers, hkv, d), dtype=torch.float32, device=q_cal.device)
    reps = (CalibReport * n_layers)()
    _check(lib.hifa4_calibrate_smooth_qk_layers(ctypes.byref(p), n_layers, n, _ptr(q_cal), _ptr(k_cal),
                                                float(alpha), _ptr(out), reps, _ptr(ws), ws_bytes,
                                                _stream(q_cal.device)), "hifa4_calibrate_smooth_qk_layers")
    return out, [{"rho_k": r.rho_k, "t_kq": r.t_kq, "branch": r.branch, "alpha_used": r.alpha_used} for r in reps]


def hifa4_quantize_qk(q, k, s=None, cu_seqlens=None, max_seqlen=None):
    """Canonical HIF4 codes of Smooth-QK'd Q and K.  Returns (q_codes uint8
    [T,Hq,D/64,32], q_meta int32 [T,Hq,D/64], k_codes, k_meta) -- meta words
    are uint32 bit patterns held in int32 tensors.  q=None quantizes K only
    (q_codes and q_meta are then None)."""
    torch = _torch()
    _require(q, torch.float16, "q")
    _require(k, torch.float16, "k")
    _require(s, torch.float32, "s")
    sh = shape_of(k if q is None else q, k, cu_seqlens, max_seqlen)
    lib = load_library()
    g = sh.head_dim // 64
    dev = k.device
    qc = qm = None
    if q is not None:
        qc = torch.empty((sh.tokens, sh.heads_q, g, 32), dtype=torch.uint8, device=dev)
        qm = torch.empty((sh.tokens, sh.heads_q, g), dtype=torch.int32, device=dev)
    kc = torch.empty((sh.tokens, sh.heads_kv, g, 32), dtype=torch.uint8, device=dev)
    km = torch.empty((sh.tokens, sh.heads_kv, g), dtype=torch.int32, device=dev)
    p = sh.problem()
    _check(lib.hifa4_quantize_qk(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(s), _ptr(qc), _ptr(qm), _ptr(kc),
                                 _ptr(km), _stream(dev)), "hifa4_quantize_qk")
    return qc, qm, kc, km


def hifa4_quantize_v(v, cu_seqlens=None, max_seqlen=None):
    """Canonical HIF4 codes of V along tokens: (codes uint8 [B, NB, Hkv, D, 32],
    meta int32 [B, NB, Hkv, D])."""
    torch = _torch()
    _require(v, torch.float16, "v")
    sh = shape_of(v, v, cu_seqlens, max_seqlen)
    lib = load_library()
    nb = (sh.max_seqlen + 63) // 64
    vc = torch.empty((sh.batch, nb, sh.heads_kv if cu_seqlens is None else v.shape[1], sh.head_dim, 32),
                     dtype=torch.uint8, device=v.device)
    sh.heads_kv = vc.shape[2]
    sh.heads_q = vc.shape[2]
    vm = torch.empty(vc.shape[:-1], dtype=torch.int32, device=v.device)
    p = sh.problem()
    _check(lib.hifa4_quantize_v(ctypes.byref(p), _ptr(v), _ptr(vc), _ptr(vm), _stream(v.device)), "hifa4_quantize_v")
    return vc, vm


class Workspace:
    """A reusable device workspace (grown on demand)."""

    def __init__(self):
        self.buf = None

    def get(self, nbytes: int, device):
        torch = _torch()
        if self.buf is None or self.buf.numel() < nbytes or self.buf.device != device:
            self.buf = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
        return self.buf


_default_ws = Workspace()


def hifa4_attention_fwd(q, k, v, s=None, cu_seqlens=None, max_seqlen=None, norm: int = NORM_PREORDER,
                        operands: int = OPERANDS_HIF4, smooth_qk: Optional[bool] = None, debug_p: bool = False,
                        out=None, lse=None, workspace: Optional[Workspace] = None, timing_events=None,
                        q_mean: bool = False, debug_heads=None, debug_tokens=None):
    """HiFA4 causal prefill forward.  Returns (o, lse) or, with debug_p,
    (o, lse, p_codes uint8 [NH,NT,NB,32], p_meta int32 [NH,NT,NB]) for the
    dump window debug_heads = (h0, NH) and debug_tokens = (t0, NT) (default:
    every head and token).  timing_events: optional three recorded
    torch.cuda.Event objects (before the pre-pass, before the attention
    kernel, after it).  q_mean: the Q-Mean auxiliary (HIF4 operands only)."""
    torch = _torch()
    for t, n in ((q, "q"), (k, "k"), (v, "v")):
        _require(t, torch.float16, n)
    _require(s, torch.float32, "s")
    sh = shape_of(q, k, cu_seqlens, max_seqlen)
    lib = load_library()
    dev = q.device
    if smooth_qk is None:
        smooth_qk = s is not None
    o = torch.empty_like(q) if out is None else out
    l = torch.empty((sh.heads_q, sh.tokens), dtype=torch.float32, device=dev) if lse is None else lse
    pc = pm = None
    h0, nh = debug_heads if debug_heads is not None else (0, 0)
    t0, nt = debug_tokens if debug_tokens is not None else (0, 0)
    if debug_p:
        nb = (sh.max_seqlen + 63) // 64
        pc = torch.zeros((nh or sh.heads_q, nt or sh.tokens, nb, 32), dtype=torch.uint8, device=dev)
        pm = torch.zeros((nh or sh.heads_q, nt or sh.tokens, nb), dtype=torch.int32, device=dev)
    ev_arr = None
    if timing_events is not None:
        ev_arr = (ctypes.c_void_p * 3)(*[e.cuda_event for e in timing_events])
    opt = FwdOptions(norm, operands, 1 if smooth_qk else 0, _ptr(pc), _ptr(pm),
                     ctypes.cast(ev_arr, ctypes.c_void_p) if ev_arr is not None else None, 1 if q_mean else 0,
                     0, h0, nh, t0, nt)
    p = sh.problem()
    need = int(lib.hifa4_workspace_bytes(ctypes.byref(p), ctypes.byref(opt)))
    ws = (workspace or _default_ws).get(need, dev)
    _check(lib.hifa4_attention_fwd(ctypes.byref(p), ctypes.byref(opt), _ptr(q), _ptr(k), _ptr(v), _ptr(s),
                                   _ptr(o), _ptr(l), _ptr(ws), ws.numel(), _stream(dev)), "hifa4_attention_fwd")
    if debug_p:
        return o, l, pc, pm
    return o, l


def hifa4_attention_fwd_noalloc(q, k, v, s=None, cu_seqlens=None, max_seqlen=None, norm: int = NORM_PREORDER,
                                operands: int = OPERANDS_HIF4, smooth_qk: Optional[bool] = None, out=None,
                                lse=None):
    """hifa4_attention_fwd with the library's static per-GPU scratch array as
    its workspace (no device allocation inside the call; at most
    NOALLOC_SCRATCH_BYTES of workspace).  Outputs are allocated here unless
    `out` and `lse` are given."""
    torch = _torch()
    for t, n in ((q, "q"), (k, "k"), (v, "v")):
        _require(t, torch.float16, n)
    _require(s, torch.float32, "s")
    sh = shape_of(q, k, cu_seqlens, max_seqlen)
    lib = load_library()
    dev = q.device
    if smooth_qk is None:
        smooth_qk = s is not None
    o = torch.empty_like(q) if out is None else out
    l = torch.empty((sh.heads_q, sh.tokens), dtype=torch.float32, device=dev) if lse is None else lse
    opt = FwdOptions(norm, operands, 1 if smooth_qk else 0, None, None, None, 0)
    p = sh.problem()
    _check(lib.hifa4_attention_fwd_noalloc(ctypes.byref(p), ctypes.byref(opt), _ptr(q), _ptr(k), _ptr(v), _ptr(s),
                                           _ptr(o), _ptr(l), _stream(dev)), "hifa4_attention_fwd_noalloc")
    return o, l


def decode_shape(q, k_codes, cu_seqlens=None, max_seqlen=None) -> Shape:
    """Problem shape of a decode step: q [B, Hq, D], K^ cache codes
    [T, Hkv, D/64, 32] (T = B * max_seqlen without cu_seqlens)."""
    if q.dim() != 3 or k_codes.dim() != 4:
        raise ValueError("decode takes q [batch, heads, dim] and k_codes [tokens, heads_kv, dim/64, 32]")
    b, hq, d = q.shape
    t, hkv = k_codes.shape[0], k_codes.shape[1]
    if cu_seqlens is None:
        if t % b:
            raise ValueError("without cu_seqlens the cache holds batch * max_seqlen tokens")
        return Shape(b, hq, hkv, d, t // b, t)
    if max_seqlen is None:
        raise ValueError("max_seqlen is required with cu_seqlens")
    _require(cu_seqlens, _torch().int32, "cu_seqlens")
    if cu_seqlens.numel() != b + 1:
        raise ValueError("cu_seqlens must hold batch + 1 entries")
    return Shape(b, hq, hkv, d, int(max_seqlen), t, cu_seqlens)


def hifa4_decode_workspace_bytes(shape: Shape) -> int:
    p = shape.problem()
    return int(load_library().hifa4_decode_workspace_bytes(ctypes.byref(p)))


def hifa4_decode_fwd(q, k_codes, k_meta, v_codes, v_meta, s=None, cu_seqlens=None, max_seqlen=None,
                     norm: int = NORM_PREORDER, smooth_qk: Optional[bool] = None, debug_p: bool = False,
                     out=None, lse=None, workspace: Optional[Workspace] = None, timing_events=None,
                     test_no_publish: bool = False):
    """One decode step over a packed HIF4 cache: q [B, Hq, D] fp16 is the query
    of each sequence's newest token; the cache is the output of
    hifa4_quantize_qk (K^, same s) and hifa4_quantize_v (V^) over the cached
    sequences.  Returns (o [B, Hq, D], lse [Hq, B]) or, with debug_p,
    (o, lse, p_codes uint8 [Hq, B, NB, 32], p_meta int32 [Hq, B, NB])."""
    torch = _torch()
    _require(q, torch.float16, "q")
    _require(k_codes, torch.uint8, "k_codes")
    _require(k_meta, torch.int32, "k_meta")
    _require(v_codes, torch.uint8, "v_codes")
    _require(v_meta, torch.int32, "v_meta")
    _require(s, torch.float32, "s")
    sh = decode_shape(q, k_codes, cu_seqlens, max_seqlen)
    nb = (sh.max_seqlen + 63) // 64
    g = sh.head_dim // 64
    if tuple(k_meta.shape) != (sh.tokens, sh.heads_kv, g) or tuple(k_codes.shape[2:]) != (g, 32):
        raise ValueError("k_codes/k_meta do not match [tokens, heads_kv, dim/64(, 32)]")
    if tuple(v_codes.shape) != (sh.batch, nb, sh.heads_kv, sh.head_dim, 32) or \
            tuple(v_meta.shape) != (sh.batch, nb, sh.heads_kv, sh.head_dim):
        raise ValueError("v_codes/v_meta do not match [batch, NB, heads_kv, dim(, 32)]")
    lib = load_library()
    dev = q.device
    if smooth_qk is None:
        smooth_qk = s is not None
    o = torch.empty_like(q) if out is None else out
    l = torch.empty((sh.heads_q, sh.batch), dtype=torch.float32, device=dev) if lse is None else lse
    pc = pm = None
    if debug_p:
        pc = torch.zeros((sh.heads_q, sh.batch, nb, 32), dtype=torch.uint8, device=dev)
        pm = torch.zeros((sh.heads_q, sh.batch, nb), dtype=torch.int32, device=dev)
    ev_arr = None
    if timing_events is not None:
        ev_arr = (ctypes.c_void_p * 3)(*[e.cuda_event for e in timing_events])
    opt = FwdOptions(norm, OPERANDS_HIF4, 1 if smooth_qk else 0, _ptr(pc), _ptr(pm),
                     ctypes.cast(ev_arr, ctypes.c_void_p) if ev_arr is not None else None, 0,
                     1 if test_no_publish else 0)
    p = sh.problem()
    need = int(lib.hifa4_decode_workspace_bytes(ctypes.byref(p)))
    ws = (workspace or _default_ws).get(need, dev)
    _check(lib.hifa4_decode_fwd(ctypes.byref(p), ctypes.byref(opt), _ptr(q), _ptr(k_codes), _ptr(k_meta),
                                _ptr(v_codes), _ptr(v_meta), _ptr(s), _ptr(o), _ptr(l), _ptr(ws), ws.numel(),
                                _stream(dev)), "hifa4_decode_fwd")
    if debug_p:
        return o, l, pc, pm
    return o, l


def hifa4_selftest_exp2(x):
    """y = fp16(2^x) through the kernels' exponential routine (x fp16 on GPU)."""
    torch = _torch()
    _require(x, torch.float16, "x")
    y = torch.empty_like(x)
    _check(load_library().hifa4_selftest_exp2(_ptr(x), _ptr(y), x.numel(), _stream(x.device)), "hifa4_selftest_exp2")
    return y
