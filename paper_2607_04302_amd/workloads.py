"""Seeded synthetic inputs for the HiFA4 prefill workloads.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic (no quantization, no smoothing, no softmax), so both the
CPU oracle and the GPU path may consume what it produces.

Recipe (identical for every consumer):
  * ``numpy.random.default_rng(seed)`` (PCG64), ``standard_normal(shape,
    dtype=float32)``; Q, then K, then V are drawn from one generator in that
    order, C-order ``[B, S, H, D]`` (varlen: ``[total, H, D]``).
  * K outliers mimic the QK-RMSNorm channel amplification of the paper
    (Section 4.1, Figures 1-3): chosen channels of K are multiplied, in fp32,
    before the single round-to-nearest-even cast to fp16.  The channels are
    drawn from a separate "model" generator so that calibration and
    evaluation data share them, as a fixed affine weight would.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    heads_q: int
    heads_kv: int
    head_dim: int
    seqlen: int                      # fixed length (ignored when varlen)
    eval_seed: int = 0
    calib_seeds: tuple = ()
    outlier_seed: Optional[int] = None      # None: fixed channel list below
    outlier_fixed: tuple = ()               # explicit channels (all kv heads)
    outliers_per_head: int = 0
    outlier_scale: float = 1.0
    alpha: float = 0.5                      # Smooth-QK exponent; 0 => off
    varlen_lengths_seed: Optional[int] = None
    varlen_range: tuple = (512, 2048)
    calib_seqlen: Optional[int] = None
    calib_from: Optional[str] = None        # reuse another workload's scales
    q_bias: float = 0.0                     # constant added to every Q element

    @property
    def varlen(self) -> bool:
        return self.varlen_lengths_seed is not None

    def seqlens(self) -> np.ndarray:
        if not self.varlen:
            return np.full(self.batch, self.seqlen, dtype=np.int64)
        lo, hi = self.varlen_range
        return np.random.default_rng(self.varlen_lengths_seed).integers(lo, hi + 1, self.batch)

    def cu_seqlens(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.seqlens())]).astype(np.int32)

    def total_tokens(self) -> int:
        return int(self.seqlens().sum())

    def causal_pairs(self) -> int:
        s = self.seqlens().astype(np.int64)
        return int((s * (s + 1) // 2).sum())

    def flops(self) -> float:
        """Algorithmic FLOPs of one forward: QK^T plus PV over causal pairs
        (diagonal included), 2 flops per multiply-add, per query head."""
        return 4.0 * self.head_dim * self.heads_q * self.causal_pairs()

    def decode_cache_bytes(self) -> int:
        """Bytes of the packed HIF4 cache one decode step reads: K^ as 36 B
        per 64 channels of every cached token and kv head, V^ as 36 B per
        64-token group of every (block, kv head, channel)."""
        s = self.seqlens().astype(np.int64)
        g = self.head_dim // 64
        k = int(s.sum()) * self.heads_kv * g * 36
        v = int(((s + 63) // 64).sum()) * self.heads_kv * self.head_dim * 36
        return k + v

    def outlier_channels(self) -> np.ndarray:
        """[Hkv, n] sorted channel indices that carry the K outlier."""
        if self.outliers_per_head == 0 and not self.outlier_fixed:
            return np.zeros((self.heads_kv, 0), dtype=np.int64)
        if self.outlier_fixed:
            return np.tile(np.array(sorted(self.outlier_fixed)), (self.heads_kv, 1))
        g = np.random.default_rng(self.outlier_seed)
        return np.stack([np.sort(g.choice(self.head_dim, self.outliers_per_head, replace=False))
                         for _ in range(self.heads_kv)])


WORKLOADS = {
    "tiny_s256": Workload("tiny_s256", 1, 1, 1, 128, 256, eval_seed=0,
                          calib_seeds=(1001, 1002, 1003, 1004),
                          outlier_fixed=(3, 17, 64, 100), outlier_scale=16.0, alpha=0.5),
    "qwen3_8b_s4096": Workload("qwen3_8b_s4096", 1, 32, 8, 128, 4096, eval_seed=0,
                               calib_seeds=tuple(range(1001, 1017)), outlier_seed=4242,
                               outliers_per_head=4, outlier_scale=16.0, alpha=0.5),
    "long_s32768": Workload("long_s32768", 1, 32, 8, 128, 32768, eval_seed=0,
                            outlier_seed=4242, outliers_per_head=4, outlier_scale=16.0,
                            alpha=0.5, calib_from="qwen3_8b_s4096"),
    "varlen_b16": Workload("varlen_b16", 16, 32, 8, 128, 0, eval_seed=1,
                           varlen_lengths_seed=0, varlen_range=(512, 2048), alpha=0.0),
    # one decode step per sequence over a 32768-token packed cache
    "decode_b8_l32768": Workload("decode_b8_l32768", 8, 32, 8, 128, 32768, eval_seed=5,
                                 outlier_seed=4242, outliers_per_head=4, outlier_scale=16.0,
                                 alpha=0.5, calib_from="qwen3_8b_s4096"),
    "wide_d256": Workload("wide_d256", 2, 16, 8, 256, 8192, eval_seed=0,
                          calib_seeds=tuple(range(1001, 1017)), outlier_seed=4243,
                          outliers_per_head=8, outlier_scale=4.0, alpha=0.5, calib_seqlen=8192),
}


def _draw(rng, shape_q, shape_kv, w: Workload):
    q = rng.standard_normal(shape_q, dtype=np.float32)
    if w.q_bias:
        q += np.float32(w.q_bias)
    k = rng.standard_normal(shape_kv, dtype=np.float32)
    v = rng.standard_normal(shape_kv, dtype=np.float32)
    ch = w.outlier_channels()
    for h in range(w.heads_kv):
        for c in ch[h]:
            k[..., h, c] *= np.float32(w.outlier_scale)
    return q.astype(np.float16), k.astype(np.float16), v.astype(np.float16)


def make_inputs(w: Workload, seed: Optional[int] = None, seqlen: Optional[int] = None,
                batch: Optional[int] = None):
    """Evaluation tensors (fp16 numpy).  Fixed length: [B,S,H,D];
    varlen: [total,H,D] plus cu_seqlens int32 [B+1]."""
    rng = np.random.default_rng(w.eval_seed if seed is None else seed)
    if w.varlen:
        t = w.total_tokens()
        q, k, v = _draw(rng, (t, w.heads_q, w.head_dim), (t, w.heads_kv, w.head_dim), w)
        return q, k, v, w.cu_seqlens()
    b = w.batch if batch is None else batch
    s = w.seqlen if seqlen is None else seqlen
    q, k, v = _draw(rng, (b, s, w.heads_q, w.head_dim), (b, s, w.heads_kv, w.head_dim), w)
    return q, k, v, None


def make_decode_inputs(w: Workload, seed: Optional[int] = None):
    """A decode step: (q [B, Hq, D], k, v, cu_seqlens or None), fp16 numpy.
    q is the query of each sequence's newest token; k and v are the cached
    sequences ([B, S, Hkv, D], or [total, Hkv, D] with cu_seqlens when
    varlen), the newest token included.  One generator draws q, then K, then V."""
    rng = np.random.default_rng(w.eval_seed if seed is None else seed)
    q = rng.standard_normal((w.batch, w.heads_q, w.head_dim), dtype=np.float32)
    if w.q_bias:
        q += np.float32(w.q_bias)
    shape = (w.total_tokens(),) if w.varlen else (w.batch, w.seqlen)
    k = rng.standard_normal(shape + (w.heads_kv, w.head_dim), dtype=np.float32)
    v = rng.standard_normal(shape + (w.heads_kv, w.head_dim), dtype=np.float32)
    ch = w.outlier_channels()
    for h in range(w.heads_kv):
        for c in ch[h]:
            k[..., h, c] *= np.float32(w.outlier_scale)
    return (q.astype(np.float16), k.astype(np.float16), v.astype(np.float16),
            w.cu_seqlens() if w.varlen else None)


def make_calibration(w: Workload, n: Optional[int] = None, seqlen: Optional[int] = None):
    """Calibration draw: one sequence per seed, stacked on a leading axis:
    q [n, S, Hq, D], k [n, S, Hkv, D] (fp16).  Same outlier channels as eval."""
    seeds = w.calib_seeds[: (len(w.calib_seeds) if n is None else n)]
    s = seqlen or w.calib_seqlen or w.seqlen
    qs, ks = [], []
    for sd in seeds:
        q, k, _ = _draw(np.random.default_rng(sd), (s, w.heads_q, w.head_dim),
                        (s, w.heads_kv, w.head_dim), w)
        qs.append(q); ks.append(k)
    return np.stack(qs), np.stack(ks)


def small_case(heads_q=2, heads_kv=1, head_dim=128, seqlens=(200,), seed=7,
               outlier_channels=(5, 77), outlier_scale=16.0, q_bias=0.0):
    """A small seeded case for parity tests (varlen layout if several lengths).
    q_bias shifts every Q element (a DC bias of the queries)."""
    w = Workload("small", len(seqlens), heads_q, heads_kv, head_dim, max(seqlens),
                 outlier_fixed=tuple(c % head_dim for c in outlier_channels) if outlier_channels else (),
                 outlier_scale=outlier_scale, q_bias=q_bias)
    rng = np.random.default_rng(seed)
    t = int(sum(seqlens))
    q, k, v = _draw(rng, (t, heads_q, head_dim), (t, heads_kv, head_dim), w)
    cu = np.concatenate([[0], np.cumsum(seqlens)]).astype(np.int32)
    return q, k, v, cu
