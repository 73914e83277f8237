#!/usr/bin/env python3
"""Throughput of the HiFA4 causal prefill forward on one MI355X.

One step = one call of hifa4_attention_fwd (K/V HIF4 pre-pass + the fused
attention kernel) over the whole Qwen3-8B-shaped S=4096 prefill (B=1, Hq=32,
Hkv=8, D=128, causal, Smooth-QK on with calibration-static scales), inputs
resident in HBM.  Prints one JSON line.

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--gpus 1]

Before the warm-up steps the forward runs untimed for 0.3 s so that the GPU
reaches steady clocks (a cold MI355X needs ~40 ms of sustained work).

The line carries the metric (effective attention TFLOP/s over causal pairs),
the fraction of the dense FP4/FP6 MFMA peak, the in-run FP16-operand variant,
the roofline of the dominant kernel (measured with HIP events on the launch
stream), and the CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP6_TFLOPS = 10066.0     # MI355X dense MXFP4/MXFP6
PEAK_FP16_TFLOPS = 2516.6     # MI355X dense FP16
PEAK_HBM_GBS = 8000.0
METRIC = "HiFA4 fwd TFLOP/s (causal) + % FP4 MFMA peak, Qwen3-8B-shape S=4096"
PAPER_CONTEXT = ("paper projects a 35.4% critical-path reduction vs BF16 from an instruction-scheduling "
                 "model of an unreleased Ascend NPU (Table 10); context only, not a target")


# The translation unit of the attention kernel: its source and the headers it
# includes.  Committed counter summaries carry this digest; a change to any of
# these files makes them stale.
ATTN_SOURCES = ("hifa4_attn.hip", "hifa4_device.h", "hifa4_internal.h", "hifa4_packed.h")


def source_digest() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2607_04302_amd", "csrc")
    for f in ATTN_SOURCES:
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def read_counters(name: str):
    """HBM traffic per dispatch from a committed rocprofv3 --pmc summary, if it
    was taken on the current kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_sha256") != source_digest():
        return None
    try:
        return float(vals["hbm_bytes_per_dispatch"])
    except (KeyError, ValueError):
        return None


# VALU issue peak: 256 CUs x 4 SIMDs x 32 fp32 lanes per clock x 2.4 GHz lane
# operations per second (78.6 T); the datasheet's 157.3 TFLOP/s fp32 vector
# peak is this rate with an FMA counted as two FLOPs.  Measured on one MI355X:
# independent v_fma_f32 / v_mul_f32 / v_add_f32 issue one wave64 instruction
# per SIMD every ~2.3 cycles (63 T lane-ops/s chip-wide); packed fp16 ops,
# conversions and v_max_f32 take ~4 cycles, v_exp_*, v_rcp_f32 and
# v_fma_mix{lo,hi}_f16 ~8, so a kernel of mixed instructions is bound by
# VALU-active cycles long before it reaches this lane-op rate.
PEAK_VALU_TLANEOPS = 256 * 4 * 32 * 2.4e9 / 1e12
SIMDS = 256 * 4
XCDS = 8


def read_sq(name: str):
    """The attention kernel's SQ counters per dispatch from a committed summary
    taken on the current kernel sources (else None): non-MFMA VALU
    instructions, and the shares of SIMD cycles with a VALU instruction
    active (SQ_ACTIVE_INST_VALU counts quad-cycles summed over waves) and with
    the matrix core busy (SQ_VALU_MFMA_BUSY_CYCLES, cycles summed over
    SIMDs), both over GRBM_GUI_ACTIVE / 8 XCDs x 1024 SIMDs."""
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_sha256") != source_digest():
        return None
    try:
        cyc = float(vals["GRBM_GUI_ACTIVE"]) / XCDS * SIMDS
        return {"valu_insts": float(vals["SQ_INSTS_VALU"]) - float(vals["SQ_INSTS_MFMA"]),
                "valu_active_share": round(4 * float(vals["SQ_ACTIVE_INST_VALU"]) / cyc, 4),
                "mfma_busy_share": round(float(vals["SQ_VALU_MFMA_BUSY_CYCLES"]) / cyc, 4)}
    except (KeyError, ValueError):
        return None


# ---------------------------------------------------------------------------
# CPU baseline: the oracle as it stands, in worker processes (one per host core
# of this process's affinity set, at most 16), one task per (sequence, query
# head), one BLAS thread per process.  The workers are fresh interpreters
# (started as child processes, never forked copies of this GPU process) that
# import numpy and the oracle only and regenerate the seeded inputs
# themselves; they get the smoothing scales the GPU used.

_ORACLE_INPUTS = {}


def _oracle_init(name):
    from paper_2607_04302_amd.workloads import WORKLOADS, make_inputs
    _ORACLE_INPUTS["w"] = WORKLOADS[name]
    _ORACLE_INPUTS["x"] = make_inputs(WORKLOADS[name])


def _oracle_task(task):
    import numpy as np
    from threadpoolctl import threadpool_limits
    from oracle import attention as oatt
    b, hh, s, want_p = task
    q, k, v, cu = _ORACLE_INPUTS["x"]
    with threadpool_limits(1):
        r = oatt.attention_fwd(q, k, v, s, cu_seqlens=cu, heads=[hh], seqs=[b], want_p=want_p)[(b, hh)]
    out = {"b": b, "h": hh, "o": r["o"].astype(np.float32), "lse": r["lse"]}
    if want_p:
        out["p_codes"], out["p_meta"] = r["p_codes"], r["p_meta"]
    return out


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def oracle_full(name, s, want_p=False, procs=None):
    """The oracle on every (sequence, query head) of workload `name`; returns
    (results keyed by (b, h), wall seconds, processes)."""
    import multiprocessing as mp
    from concurrent.futures import ProcessPoolExecutor
    from paper_2607_04302_amd.workloads import WORKLOADS
    w = WORKLOADS[name]
    n_seq = w.batch
    tasks = [(b, hh, s, want_p) for b in range(n_seq) for hh in range(w.heads_q)]
    procs = procs or min(16, len(os.sched_getaffinity(0)))
    # the oracle allocates and frees large temporaries per block: keep freed
    # memory in each worker's heap (glibc settings, read at the worker's start)
    # instead of returning it to the kernel and faulting it in again
    os.environ.setdefault("MALLOC_MMAP_THRESHOLD_", str(1 << 30))
    os.environ.setdefault("MALLOC_TRIM_THRESHOLD_", str(1 << 31))
    # one BLAS thread per worker from its start (no idle thread pools spinning)
    saved = {v: os.environ.get(v) for v in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")}
    for v in saved:
        os.environ[v] = "1"
    t0 = time.perf_counter()
    # a worker that dies makes the executor raise (BrokenProcessPool) instead of waiting
    with ProcessPoolExecutor(procs, mp_context=mp.get_context("spawn"), initializer=_oracle_init,
                             initargs=(name,)) as pool:
        res = list(pool.map(_oracle_task, tasks, timeout=600))
    dt = time.perf_counter() - t0
    for v, x in saved.items():
        if x is None:
            os.environ.pop(v, None)
        else:
            os.environ[v] = x
    return {(r["b"], r["h"]): r for r in res}, dt, procs


def cpu_baseline(headline, s_by_name):
    """The oracle timed in full on the tiny, the headline and the batched
    varlen workloads (wall time of the worker pool, including each worker's
    input generation); the headline result is kept (with its P^ codes) for
    the parity maxima of the GPU run."""
    from paper_2607_04302_amd.workloads import WORKLOADS
    out = {}
    keep = None
    for name in ("tiny_s256", headline, "varlen_b16"):
        res, dt, procs = oracle_full(name, s_by_name.get(name), want_p=(name == headline))
        w = WORKLOADS[name]
        out[name] = {"seconds": round(dt, 2), "value": w.flops() / dt / 1e12, "processes": procs,
                     "tasks": len(res)}
        if name == headline:
            keep = res
    hl = out[headline]
    base = {"value": hl["value"], "unit": "TFLOP/s", "cores": hl["processes"], "kind": "oracle",
            "sample": f"{headline} in full: every query head and row ({hl['tasks']} (sequence, head) tasks), "
                      f"{hl['seconds']} s wall on {hl['processes']} worker processes of one BLAS thread each",
            "cpu_model": cpu_model(), "affinity_cores": len(os.sched_getaffinity(0)),
            "blas_threads_per_process": 1,
            "configs": {k: {"seconds": v["seconds"], "value": v["value"], "unit": "TFLOP/s"} for k, v in out.items()}}
    return base, keep


def parity_maxima(h, torch, np, w, q, k, v, s_oracle, ref):
    """The headline forward (debug dump on, the oracle's own smoothing
    scales) against the oracle's full result: P^ group mismatches over every
    (head, row, visible block), O max-abs and max-rel error, LSE max-abs."""
    res = h.hifa4_attention_fwd(q, k, v, torch.from_numpy(s_oracle).to(q.device) if s_oracle is not None else None,
                                debug_p=True)
    torch.cuda.synchronize()
    o = res[0].reshape(-1, w.heads_q, w.head_dim).float().cpu().numpy()
    lse = res[1].cpu().numpy()
    S = w.seqlen
    nb = (S + 63) // 64
    vis = (np.arange(nb)[None, :] <= (np.arange(S) // 64)[:, None])
    mism = groups = 0
    oa = orr = la = 0.0
    for (b, hh), r in ref.items():
        t = slice(b * S, (b + 1) * S)
        pc = res[2][hh, t].cpu().numpy()
        pm = res[3][hh, t].cpu().numpy().view(np.uint32)
        bad = (pc != r["p_codes"]).any(-1) | (pm != r["p_meta"])
        mism += int((bad & vis).sum())
        groups += int(vis.sum())
        ro = r["o"].astype(np.float64)
        err = np.abs(o[t, hh] - ro)
        oa = max(oa, float(err.max()))
        orr = max(orr, float((err / np.maximum(np.abs(ro), 1e-2)).max()))
        la = max(la, float(np.abs(lse[hh, t] - r["lse"]).max()))
    del res
    torch.cuda.empty_cache()
    return {"p_groups_compared": groups, "p_group_mismatches": mism, "o_max_abs": oa,
            "o_max_rel_above_1e-2": orr, "lse_max_abs": la,
            "basis": "every query head and row of the headline workload, oracle scales s"}


def config_report(h, torch, np, name, ws):
    """Throughput of the HiFA4 forward on another workload (inputs resident,
    Smooth-QK scales from its calibration draw via the GPU calibration call;
    0.2 s of back-to-back calls settle the clocks before the timed calls),
    with the pre-pass / attention-kernel split from a separate pass of the
    library's events; for the wide-head workload also the inconsistent
    normalizer and its eps, on the GPU and from the oracle on sampled rows."""
    from paper_2607_04302_amd.workloads import WORKLOADS, make_calibration, make_inputs
    w = WORKLOADS[name]
    dev = torch.device("cuda:0")
    qn, kn, vn, cun = make_inputs(w)
    q, k, v = (torch.from_numpy(x).to(dev) for x in (qn, kn, vn))
    cu = None if cun is None else torch.from_numpy(cun).to(dev)
    s = sn = None
    if w.alpha > 0:
        src = WORKLOADS[w.calib_from] if w.calib_from else w
        qc, kc = make_calibration(src)
        s, _ = h.hifa4_calibrate_smooth_qk(torch.from_numpy(qc).to(dev), torch.from_numpy(kc).to(dev), w.alpha)
        sn = s.cpu().numpy()
        del qc, kc
    flops = w.flops()
    max_s = int(w.seqlens().max())
    steps = max(3, min(50, int(2e13 / flops)))
    kw = dict(cu_seqlens=cu, max_seqlen=max_s, workspace=ws)

    def run(norm, n):
        # back-to-back calls until the clocks have settled on this workload
        # (the host work between workloads lets them drop), then the timed calls
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < 0.2:
            for _ in range(4):
                h.hifa4_attention_fwd(q, k, v, s, norm=norm, **kw)
            torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(n):
            res = h.hifa4_attention_fwd(q, k, v, s, norm=norm, **kw)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3 / n, res

    def split(norm, n):
        # median pre-pass and attention-kernel times from the library's events
        # (a separate pass: the event markers add gaps of their own)
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n)]
        for trio in evs:
            for e in trio:
                e.record()
        torch.cuda.synchronize()
        for i in range(n):
            h.hifa4_attention_fwd(q, k, v, s, norm=norm, timing_events=evs[i], **kw)
        torch.cuda.synchronize()
        pre = sorted(e[0].elapsed_time(e[1]) for e in evs)[n // 2]
        att = sorted(e[1].elapsed_time(e[2]) for e in evs)[n // 2]
        return {"kv_prepass": round(pre, 4), "attention": round(att, 4)}

    ms, (o, lse) = run(h.NORM_PREORDER, steps)
    kern = split(h.NORM_PREORDER, min(steps, 10))
    tf = flops / (ms * 1e-3) / 1e12
    out = {"workload": name, "batch": w.batch, "heads_q": w.heads_q, "heads_kv": w.heads_kv, "head_dim": w.head_dim,
           "seqlen": (f"{w.varlen_range[0]}..{w.varlen_range[1]}" if w.varlen else w.seqlen),
           "smooth_qk": s is not None, "gflop_per_step": round(flops / 1e9, 3), "steps": steps,
           "ms_per_step": round(ms, 4), "value": round(tf, 2), "unit": "TFLOP/s",
           "pct_fp4_peak": round(100.0 * tf / PEAK_FP6_TFLOPS, 3), "kernels_ms": kern,
           "attention_kernel_pct_fp4_peak": round(100.0 * flops / (kern["attention"] * 1e-3) / 1e12
                                                  / PEAK_FP6_TFLOPS, 3)}
    if name == "wide_d256":
        msi, (oi, lsei) = run(h.NORM_INCONSISTENT, steps)
        eps = torch.expm1(lse.double() - lsei.double()).cpu().numpy()
        from oracle import attention as oatt
        rows = [64, 2047, 4096, 8191]
        heads = [3]
        rc = oatt.attention_fwd(qn, kn, vn, sn, heads=heads, rows=rows, seqs=[0])
        rm = oatt.attention_fwd(qn, kn, vn, sn, heads=heads, rows=rows, seqs=[0], norm="inconsistent")
        eps_o = np.expm1(rc[(0, 3)]["lse"] - rm[(0, 3)]["lse"])
        eps_g = eps[3, rows]
        out["inconsistent_variant"] = {
            "ms_per_step": round(msi, 4), "eps_row_median": float(np.median(eps)),
            "eps_row_frac_negative": float((eps < 0).mean()),
            "eps_sampled_rows": {"rows": rows, "head": 3, "gpu": [float(x) for x in eps_g],
                                 "oracle": [float(x) for x in eps_o]}}
    del q, k, v, o, lse
    torch.cuda.empty_cache()
    return out


def decode_report(h, torch, np, ws, steps=50):
    """One decode step per sequence over the packed HIF4 cache of the
    8 x 32768-token decode workload (Qwen3-8B heads, Smooth-QK scales from
    the Qwen3-shaped calibration draw): the cache is built once on the GPU,
    then back-to-back decode calls are timed with HIP events recorded by the
    library (before the query quantization, after the score kernel, after the
    merge).  HBM roofline on the bytes of the packed cache a step reads."""
    from paper_2607_04302_amd.workloads import WORKLOADS, make_calibration, make_decode_inputs
    w = WORKLOADS["decode_b8_l32768"]
    dev = torch.device("cuda:0")
    qn, kn, vn, _ = make_decode_inputs(w)
    qc, kc = make_calibration(WORKLOADS[w.calib_from])
    s, _ = h.hifa4_calibrate_smooth_qk(torch.from_numpy(qc).to(dev), torch.from_numpy(kc).to(dev), w.alpha)
    del qc, kc
    q = torch.from_numpy(qn).to(dev)
    k = torch.from_numpy(kn).to(dev)
    v = torch.from_numpy(vn).to(dev)
    _, _, kcode, kmeta = h.hifa4_quantize_qk(None, k, s)
    vcode, vmeta = h.hifa4_quantize_v(v)
    del k, v
    torch.cuda.empty_cache()
    out = torch.empty_like(q)
    lse = torch.empty((w.heads_q, w.batch), dtype=torch.float32, device=dev)
    kw = dict(out=out, lse=lse, workspace=ws)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    for trio in evs:
        for e in trio:
            e.record()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < 0.2:
        for _ in range(10):
            h.hifa4_decode_fwd(q, kcode, kmeta, vcode, vmeta, s, **kw)
        torch.cuda.synchronize()
    # the step time: back-to-back calls between one pair of events
    da, db = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    da.record()
    for _ in range(steps):
        h.hifa4_decode_fwd(q, kcode, kmeta, vcode, vmeta, s, **kw)
    db.record()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / steps
    dev_ms = da.elapsed_time(db) / steps
    # the split between scores plus splits and the merge, from the library's
    # events inside each call (a separate pass: those events add their own
    # gaps)
    for i in range(steps):
        h.hifa4_decode_fwd(q, kcode, kmeta, vcode, vmeta, s, timing_events=evs[i], **kw)
    torch.cuda.synchronize()
    first = sum(evs[i][0].elapsed_time(evs[i][1]) for i in range(steps)) / steps
    second = sum(evs[i][1].elapsed_time(evs[i][2]) for i in range(steps)) / steps
    # the same step captured once as a HIP graph and replayed back to back
    # (the library's launches carry no memsets, so they capture as they are)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        h.hifa4_decode_fwd(q, kcode, kmeta, vcode, vmeta, s, **kw)
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        h.hifa4_decode_fwd(q, kcode, kmeta, vcode, vmeta, s, **kw)
    for _ in range(10):
        graph.replay()
    ga, gb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ga.record()
    for _ in range(steps):
        graph.replay()
    gb.record()
    torch.cuda.synchronize()
    graph_ms = ga.elapsed_time(gb) / steps
    del graph
    cache = w.decode_cache_bytes()
    gbs = cache / (dev_ms * 1e-3) / 1e9
    res = {"workload": w.name, "batch": w.batch, "heads_q": w.heads_q, "heads_kv": w.heads_kv,
           "head_dim": w.head_dim, "cached_tokens_per_sequence": w.seqlen, "smooth_qk": True,
           "cache_bytes": cache, "fp16_cache_bytes": 2 * 2 * w.total_tokens() * w.heads_kv * w.head_dim,
           "steps": steps, "ms_per_step": round(dev_ms, 4), "wall_ms_per_step": round(wall, 4),
           "graph_replay_ms_per_step": round(graph_ms, 4),
           "kernels_ms": {"scores_and_splits": round(first, 4), "merge": round(second, 4),
                          "basis": "library events inside each call, a separate pass"},
           "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                        "frac": round(gbs / PEAK_HBM_GBS, 4),
                        "basis": "packed K^ and V^ cache bytes per step / device time per step of "
                                 "back-to-back calls"}}
    del q, kcode, kmeta, vcode, vmeta, out, lse
    torch.cuda.empty_cache()
    return res


def p_only_study(h, torch, np, args, q, k, v, out16, ws):
    """The P-only local operator (Q, K, V fp16, only P quantized) on the same
    inputs, with the consistent (P-Reordering) and the inconsistent
    normalizer: row-wise cosine similarity and output-norm ratio against the
    FP16 reference output, and the per-row eps = l_con/l_mis - 1 =
    exp(LSE_con - LSE_mis) - 1 (Theorem 1) as a distribution."""
    ref = out16.float().reshape(-1, out16.shape[-1])
    res = {}
    lses = {}
    for name, norm in (("consistent", h.NORM_PREORDER), ("inconsistent", h.NORM_INCONSISTENT)):
        wall, _, att, o, lse = time_variant(h, torch, args, q, k, v, None, norm, h.OPERANDS_P_ONLY,
                                            max(5, args.steps // 10), 2, ws)
        x = o.float().reshape(-1, o.shape[-1])
        cos = (x * ref).sum(1) / (x.norm(dim=1) * ref.norm(dim=1)).clamp_min(1e-30)
        ratio = x.norm(dim=1) / ref.norm(dim=1).clamp_min(1e-30)
        res[name] = {"ms_per_step": round(wall, 4), "attention_ms": round(att, 4),
                     "cos_mean": round(float(cos.mean()), 6), "cos_min": round(float(cos.min()), 6),
                     "norm_ratio_median": round(float(ratio.median()), 6),
                     "norm_ratio_mean": round(float(ratio.mean()), 6)}
        lses[name] = lse
    eps = torch.expm1(lses["consistent"].double() - lses["inconsistent"].double()).cpu().numpy().ravel()
    edges = np.array([-0.2, -0.1, -0.05, -0.02, -0.01, -0.005, 0.0, 0.005, 0.01, 0.02, 0.05])
    counts, _ = np.histogram(np.clip(eps, edges[0], edges[-1]), bins=edges)
    res["eps_row"] = {"median": float(np.median(eps)), "p10": float(np.percentile(eps, 10)),
                      "p90": float(np.percentile(eps, 90)), "frac_negative": float((eps < 0).mean()),
                      "hist_edges": edges.tolist(), "hist_counts": counts.tolist()}
    return res


def settle_clocks(h, torch, q, k, v, s, ws, seconds=0.3):
    """Untimed calls of the measured forward until the GPU has run it for
    `seconds` of wall time.  A cold MI355X raises its clocks over the first
    ~40 ms of sustained work (a call at S=4096 takes ~1.3x its steady-state
    time at first), so the timed steps start from steady clocks whatever the
    warm-up count.  Returns the number of calls."""
    n = 0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(10):
            h.hifa4_attention_fwd(q, k, v, s, workspace=ws)
        torch.cuda.synchronize()
        n += 10
    return n


def time_variant(h, torch, args, q, k, v, s, norm, operands, steps, warmup, ws, q_mean=False):
    """Settle the clocks on this variant, run warmup + steps back-to-back
    calls; returns (ms_per_step wall of the plain calls, per-step prepass ms,
    per-step attention ms, O, LSE), the two kernel times from a second pass
    of steps calls with HIP events recorded by the library on the launch
    stream around each kernel."""
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    for trio in evs:          # create the underlying HIP events
        for e in trio:
            e.record()
    torch.cuda.synchronize()
    kw = dict(s=s, norm=norm, operands=operands, smooth_qk=s is not None and operands == h.OPERANDS_HIF4,
              workspace=ws, q_mean=q_mean)
    out = torch.empty_like(q)
    lse = torch.empty((q.shape[2], q.shape[0] * q.shape[1]), dtype=torch.float32, device=q.device)
    # back-to-back calls of this variant until the clocks have settled again
    # (host work between variants lets them drop), then the warm-up steps
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < 0.2:
        for _ in range(5):
            h.hifa4_attention_fwd(q, k, v, out=out, lse=lse, **kw)
        torch.cuda.synchronize()
    for _ in range(warmup):
        h.hifa4_attention_fwd(q, k, v, out=out, lse=lse, **kw)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        h.hifa4_attention_fwd(q, k, v, out=out, lse=lse, **kw)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / steps
    # the split between the pre-pass and the attention kernel, from the
    # library's events inside each call, in a separate pass (the event
    # markers between the two launches add gaps of their own)
    for i in range(steps):
        h.hifa4_attention_fwd(q, k, v, out=out, lse=lse, timing_events=evs[i], **kw)
    torch.cuda.synchronize()
    pre = [evs[i][0].elapsed_time(evs[i][1]) for i in range(steps)]
    att = [evs[i][1].elapsed_time(evs[i][2]) for i in range(steps)]
    return wall, sum(pre) / steps, sum(att) / steps, out, lse


def valu_roofline(sq, att_ms):
    """The attention kernel against VALU issue: non-MFMA VALU instructions per
    dispatch (SQ counters) x 64 lanes / the live mean kernel time, against
    PEAK_VALU_TLANEOPS; with the VALU-active and MFMA-busy shares of SIMD
    cycles from the same counters (the VALU-active share is the bound that
    binds: most of the kernel's instructions issue at 4 or 8 cycles)."""
    if sq is None:
        return None
    achieved = sq["valu_insts"] * 64 / (att_ms * 1e-3) / 1e12
    return {"bound": "alu", "achieved": round(achieved, 2), "peak": round(PEAK_VALU_TLANEOPS, 2),
            "unit": "T VALU lane-ops/s", "frac": round(achieved / PEAK_VALU_TLANEOPS, 4),
            "valu_instructions_per_dispatch": sq["valu_insts"],
            "valu_active_share_of_simd_cycles": sq["valu_active_share"],
            "mfma_busy_share_of_simd_cycles": sq["mfma_busy_share"]}


def call_distribution(h, torch, np, q, k, v, s, ws, steps=100, cold_steps=20):
    """Device time per call (the library's events before the pre-pass and
    after the attention kernel): median, p10 and p90 over back-to-back calls
    with warm caches, then the median over calls that each follow a 512 MiB
    scrub write (L2 and the 256 MB MALL evicted)."""
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    for trio in evs:
        for e in trio:
            e.record()
    out = torch.empty_like(q)
    lse = torch.empty((q.shape[2], q.shape[0] * q.shape[1]), dtype=torch.float32, device=q.device)
    kw = dict(s=s, smooth_qk=s is not None, workspace=ws, out=out, lse=lse)
    for _ in range(10):
        h.hifa4_attention_fwd(q, k, v, **kw)
    torch.cuda.synchronize()
    for i in range(steps):
        h.hifa4_attention_fwd(q, k, v, timing_events=evs[i], **kw)
    torch.cuda.synchronize()
    warm = np.array([e[0].elapsed_time(e[2]) for e in evs]) * 1e3
    scrub = torch.empty(512 << 20, dtype=torch.uint8, device=q.device)
    cold = []
    for i in range(cold_steps):
        scrub.fill_(i & 255)
        h.hifa4_attention_fwd(q, k, v, timing_events=evs[i], **kw)
        torch.cuda.synchronize()
        cold.append(evs[i][0].elapsed_time(evs[i][2]) * 1e3)
    del scrub
    return {"unit": "us", "warm_median": round(float(np.median(warm)), 2),
            "warm_p10": round(float(np.percentile(warm, 10)), 2), "warm_p90": round(float(np.percentile(warm, 90)), 2),
            "cold_median": round(float(np.median(cold)), 2), "warm_steps": steps, "cold_steps": cold_steps}


def observed_sclk(h, torch, q, k, v, s, ws, seconds=1.0):
    """GPU core clock read with rocm-smi (a child process) half way through a
    second of back-to-back forward calls; None if the tool is unavailable."""
    import re
    import subprocess
    import threading
    box = {}

    def probe():
        time.sleep(seconds / 2)
        try:
            import shutil
            tool = shutil.which("rocm-smi") or "/opt/rocm/bin/rocm-smi"
            r = subprocess.run([tool, "--showclocks"], capture_output=True, text=True, timeout=20)
            m = re.search(r"sclk[^(]*\((\d+)\s*Mhz\)", r.stdout, re.IGNORECASE)
            box["mhz"] = int(m.group(1)) if m else None
        except Exception:
            box["mhz"] = None

    t = threading.Thread(target=probe)
    t.start()
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(10):
            h.hifa4_attention_fwd(q, k, v, s, workspace=ws)
        torch.cuda.synchronize()
    t.join()
    return box.get("mhz")


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="qwen3_8b_s4096")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-variants", action="store_true", help="time only the HiFA4 path")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the throughput of the other workloads (tiny, long, varlen, wide)")
    ap.add_argument("--no-decode", action="store_true", help="skip the decode step over the packed cache")
    ap.add_argument("--no-clock-query", action="store_true",
                    help="skip the rocm-smi clock reading (a child process); for runs under a profiler, whose "
                         "preloaded library has initialised the GPU in the process the child is forked from")
    ap.add_argument("--decode-only", action="store_true",
                    help="only time the decode step (for profiling its kernels) and print its report")
    ap.add_argument("--issue-probe", action="store_true",
                    help="only run the instruction issue-cost probe (built with the library) and print its lines")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB five times (the reference kernel that "
                         "scales HBM traffic counters) and exit")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on exactly one GPU: the HiFA4 forward shards by (batch, KV head) with no "
              "cross-GPU exchange, and this build measures one GPU's share.  Use --gpus 1.", file=sys.stderr)
        sys.exit(2)

    if args.issue_probe:
        import subprocess
        probe = os.path.join(ROOT, "paper_2607_04302_amd", "issue_probe")
        if not os.path.exists(probe):
            print("issue_probe not built (python -m paper_2607_04302_amd.build)", file=sys.stderr)
            sys.exit(1)
        sys.exit(subprocess.run([probe]).returncode)
    import numpy as np
    import torch
    if args.copy_probe:
        n = args.copy_probe << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n, "copies": 5}), flush=True)
        return
    import paper_2607_04302_amd as h
    from paper_2607_04302_amd.workloads import WORKLOADS, make_calibration, make_inputs

    h.load_library()
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    if args.decode_only:
        print(json.dumps({"decode": decode_report(h, torch, np, h.Workspace(), steps=args.steps)}), flush=True)
        return
    w = WORKLOADS[args.workload]
    if w.varlen:
        print("bench.py times fixed-length workloads", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    qn, kn, vn, _ = make_inputs(w)
    q = torch.from_numpy(qn).to(dev)
    k = torch.from_numpy(kn).to(dev)
    v = torch.from_numpy(vn).to(dev)
    s = None
    sn = None
    calib = None
    if w.alpha > 0:
        src = WORKLOADS[w.calib_from] if w.calib_from else w
        qc, kc = make_calibration(src)
        qcd, kcd = torch.from_numpy(qc).to(dev), torch.from_numpy(kc).to(dev)
        torch.cuda.synchronize()
        tc = time.perf_counter()
        s, rep = h.hifa4_calibrate_smooth_qk(qcd, kcd, w.alpha)     # synchronizes
        tc = time.perf_counter() - tc
        del qc, kc, qcd, kcd
        sn = s.cpu().numpy()
        calib = {"n_calib": len(src.calib_seeds), "alpha": w.alpha, "rho_k": round(rep["rho_k"], 3),
                 "t_kq": round(rep["t_kq"], 3), "seconds": round(tc, 4)}
    torch.cuda.synchronize()
    flops = w.flops()
    ws = h.Workspace()

    settle = settle_clocks(h, torch, q, k, v, s, ws)
    wall, pre_ms, att_ms, out, lse = time_variant(h, torch, args, q, k, v, s, h.NORM_PREORDER, h.OPERANDS_HIF4,
                                                  args.steps, args.warmup, ws)
    value = flops / (wall * 1e-3) / 1e12
    att_tflops = flops / (att_ms * 1e-3) / 1e12
    traffic = read_counters(f"attn_hif4_{w.name}_counters.txt")
    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp6",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "heads_q": w.heads_q, "heads_kv": w.heads_kv,
                   "head_dim": w.head_dim, "seqlen": w.seqlen, "causal": True, "smooth_qk": s is not None,
                   "norm": "p_reordering", "operands": "HIF4 (FP6 E2M3 MFMA operands, fp32 accumulate, fp16 softmax)",
                   "gflop_per_step": round(flops / 1e9, 3), "calibration": calib},
        "pct_fp4_peak": round(100.0 * value / PEAK_FP6_TFLOPS, 3),
        "kernels_ms": {"kv_prepass": round(pre_ms, 4), "attention": round(att_ms, 4)},
        "roofline": {"bound": "mfma", "achieved": round(att_tflops, 2), "peak": PEAK_FP6_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(att_tflops / PEAK_FP6_TFLOPS, 5),
                     "traffic": traffic, "kernel": f"k_attn_hif4<G={w.head_dim // 64},preorder>",
                     "source_sha256": source_digest()},
        "paper_context": PAPER_CONTEXT,
        "clock_settle_calls": settle,
        "valu_roofline": valu_roofline(read_sq(f"attn_hif4_{w.name}_sq_counters.txt"), att_ms),
        "call_device_time": call_distribution(h, torch, np, q, k, v, s, ws),
        "sclk_mhz_during_calls": None if args.no_clock_query else observed_sclk(h, torch, q, k, v, s, ws),
    }
    if not args.no_variants:
        wall16, pre16, att16, out16, _ = time_variant(h, torch, args, q, k, v, None, h.NORM_PREORDER,
                                                      h.OPERANDS_FP16, args.steps, args.warmup, ws)
        v16 = flops / (wall16 * 1e-3) / 1e12
        result["fp16_variant"] = {"value": round(v16, 2), "unit": "TFLOP/s", "ms_per_step": round(wall16, 4),
                                  "pct_fp16_peak": round(100.0 * v16 / PEAK_FP16_TFLOPS, 3),
                                  "kernels_ms": {"kv_prepass": round(pre16, 4), "attention": round(att16, 4)}}
        result["speedup_vs_fp16"] = round(wall16 / wall, 4)
        walli, _, atti, outi, lsei = time_variant(h, torch, args, q, k, v, s, h.NORM_INCONSISTENT,
                                                  h.OPERANDS_HIF4, max(5, args.steps // 5), 2, ws)
        # per-row eps = l_con/l_mis - 1 = exp(LSE_con - LSE_mis) - 1 (Theorem 1)
        eps = torch.expm1(lse.double() - lsei.double()).cpu().numpy()
        result["inconsistent_variant"] = {"ms_per_step": round(walli, 4),
                                          "eps_row_median": float(np.median(eps)),
                                          "eps_row_frac_negative": float((eps < 0).mean())}
        wallq, preq, attq, outq, _ = time_variant(h, torch, args, q, k, v, s, h.NORM_PREORDER, h.OPERANDS_HIF4,
                                                  max(5, args.steps // 5), 2, ws, q_mean=True)
        result["qmean_variant"] = {"value": round(flops / (wallq * 1e-3) / 1e12, 2), "unit": "TFLOP/s",
                                   "ms_per_step": round(wallq, 4),
                                   "kernels_ms": {"kv_prepass": round(preq, 4), "attention": round(attq, 4)}}
        del outq
        result["p_only_study"] = p_only_study(h, torch, np, args, q, k, v, out16, ws)
        # Fidelity diagnostic (not gating): rel-L2 of HiFA4 O against the FP16 variant.
        diff = (out.float() - out16.float()).norm() / out16.float().norm()
        result["rel_l2_vs_fp16_variant"] = round(float(diff), 5)
        del out16, outi, lsei
    if not args.no_configs:
        del out, lse
        torch.cuda.empty_cache()
        result["other_configs"] = [config_report(h, torch, np, name, ws)
                                   for name in ("tiny_s256", "long_s32768", "varlen_b16", "wide_d256")]
    if not args.no_decode:
        result["decode"] = decode_report(h, torch, np, ws)
    if not args.no_cpu_baseline:
        s_by = {w.name: sn}
        tw = WORKLOADS["tiny_s256"]
        qc, kc = make_calibration(tw)
        st, _ = h.hifa4_calibrate_smooth_qk(torch.from_numpy(qc).to(dev), torch.from_numpy(kc).to(dev), tw.alpha)
        s_by["tiny_s256"] = st.cpu().numpy()
        result["cpu_baseline"], ref = cpu_baseline(w.name, s_by)
        result["parity"] = parity_maxima(h, torch, np, w, q, k, v, sn, ref)
        del ref
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
