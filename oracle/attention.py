"""The HiFA4 (C4V16) causal prefill forward, step by step.

Paper: Algorithm 1 (C4V16-Aux), with the Q-Mean steps optional (qmean.py);
Background,
"FlashAttention tiling" (online softmax); Section 4.5 (P-Reordering,
Theorem 1, fused normalizer [V|1]); "P-Reordering under online softmax";
Appendix C (quantized tensors, FP16 operations, GQA).

Readings fixed here (the paper is silent on them):
  * logical KV block = 64 keys = one P group, processed in ascending order;
    blocks are aligned to each sequence's first token;
  * Q~ and K~ are HIF4-quantized along the head dimension (64-channel groups),
    V along tokens (64 tokens of one channel; a partial last group is zero
    padded), P along the 64 keys of a block -- every group lies along the
    contraction axis of its GEMM;
  * scores (Algorithm 1's S = Q^K^T/sqrt(d), computed on the HIF4 matrix
    unit): per 64-channel group g the term t_g = (dequantized Q^ group) .
    (dequantized K^ group) is exact (a block-scaled product forms each
    group's dot and applies both block scales without rounding; t_g has at
    most 22 significant bits); the groups are summed in fp32 in contraction
    order, S_acc = fp32(fp32(t_0 + t_1) + t_2) ..., each addition rounded
    once (nearest even); then the score scale c = fp32(log2(e)/sqrt(D)) is
    one fp32 multiply, and the product is converted to the fp16 the softmax
    works in: S2 = fp16(fp32(S_acc * c)).  With Q-Mean the correction
    mu_i * kappa_j (Algorithm 1's added term, after the group terms) is added
    to S_acc with one rounding before the scale.  The softmax runs in base 2
    (2^(S2-m) equals exp(S/sqrt(D) - m') exactly in real arithmetic);
  * running max m and the weights are fp16: m_new = max(m, rowmax S2),
    x = fp16(S2 - m_new), P16 = E(x), r = E(fp16(m - m_new));
  * P-Reordering: P^ = HIF4(P16 over the block), O <- r*O + P^ V^,
    l <- r*l + rowsum(P^); the inconsistent (Direct) variant keeps
    l <- r*l + rowsum(P16) (Theorem 1's partition sum Z);
  * O and l are accumulated in float64 here (fp32 on the GPU; the paper keeps
    l in FP16, which cannot hold sums past 2048 -- a documented deviation);
  * finalize: O = fp16(fp32(O / l)); LSE = m*ln2 + ln(l) (natural log, fp32).
  * causal: key j is visible to query i (same sequence) iff j <= i.

``arith="exact"`` runs the same loop with no quantization and no fp16
rounding (float64 scores, exp and state), for the brute-force pin.
"""
from __future__ import annotations

import math

import numpy as np

from . import hif4
from .smooth import apply as smooth_apply
from . import qmean as _qmean
from .qmean import key_sums, token_mean, zero_mean
from .softmax16 import exp2_fp16, sub_fp16

BLOCK = 64
LN2 = math.log(2.0)


def score_scale(head_dim: int) -> np.float32:
    """c = fp32(log2(e) / sqrt(D)), computed in float64 and rounded once."""
    return np.float32(math.log2(math.e) / math.sqrt(head_dim))


def quantize_rows(x):
    """HIF4 along the last axis (groups of 64 consecutive channels)."""
    lead, d = x.shape[:-1], x.shape[-1]
    f = hif4.quantize(np.asarray(x, np.float64).reshape(*lead, d // 64, 64))
    return f


def quantize_tokens(v):
    """HIF4 of V along tokens: v [L, D] -> groups of 64 tokens per channel,
    zero padded to a multiple of 64.  Returns (fields over [D, L/64, 64],
    vhat [Lpad, D])."""
    L, d = v.shape
    lp = -(-L // BLOCK) * BLOCK
    vp = np.zeros((lp, d), np.float64)
    vp[:L] = v.astype(np.float64)
    g = vp.T.reshape(d, lp // BLOCK, BLOCK)
    f = hif4.quantize(g)
    vhat = f["xhat"].reshape(d, lp).T.copy()
    return f, vhat


def unit_operands(fields):
    """The Q operand values +-u*2^-sh of HIF4 groups: the dequantized values
    divided by b/4 (exact), from the stored fields."""
    shift = (np.repeat(fields["e2"], 8, axis=-1).astype(np.int64)
             + np.repeat(fields["e3"], 4, axis=-1))
    u = fields["u"].astype(np.float64)
    return np.where(fields["sign"], -u, u) * np.exp2(-shift.astype(np.float64))


def scores_hif4(q_op, q_base, khat, head_dim, corr=None):
    """S2 [n, L] (fp16) from the Q operand values q_op [n, D] (+-u*2^-sh),
    the Q group bases q_base [n, D/64] (E6M2 values) and the dequantized K^
    [L, D] (float64).

    t_g = (q_op_g * q_base_g/4) . khat_g, the exact dot of the dequantized
    groups (float64 holds it exactly; it is also exact in fp32).  S_acc is
    their fp32 sum in group order, each addition rounded once; with Q-Mean,
    corr = (mu [n] fp16, kappa [L] fp32) and S_acc = fp32(S_acc + mu*kappa)
    (the exact product added with one rounding).  S2 = fp16(fp32(S_acc*c))."""
    c = score_scale(head_dim)
    acc = None
    for g in range(head_dim // 64):
        sl = slice(64 * g, 64 * g + 64)
        qdq = q_op[:, sl] * (np.asarray(q_base, np.float64)[:, g:g + 1] / 4.0)    # dequantized Q^ group
        t = qdq @ khat[:, sl].T                                                    # exact
        t32 = t.astype(np.float32)
        assert np.array_equal(t32.astype(np.float64), t), "group term not exact in fp32"
        acc = t32 if acc is None else (acc + t32)                                  # fp32 RNE
    if corr is not None:
        acc = _qmean.add_correction(acc, *corr)
    return (acc * c).astype(np.float16)


def scores_fp16(q, k, head_dim):
    """FP16-operand variant: fp32 dot of the fp16 operands; times c in fp32,
    then to fp16."""
    c = score_scale(head_dim)
    s = (q.astype(np.float64) @ k.astype(np.float64).T).astype(np.float32)
    return (s * c).astype(np.float32).astype(np.float16)


def online_softmax(s2, vop, rows, length, quantize_p, want_p=False, arith="contract"):
    """Algorithm 1's tile loop for the query rows ``rows`` of one (sequence,
    head).  s2: [n, length] scores of those rows (fp16, or float64 when
    arith == "exact"); vop: [Lpad, D] value operand (V^ or V) in float64."""
    n, d = len(rows), vop.shape[1]
    nblk = -(-length // BLOCK)
    exact = arith == "exact"
    m = np.full(n, -np.inf, np.float64 if exact else np.float16)
    o = np.zeros((n, d))
    l_con = np.zeros(n)
    l_mis = np.zeros(n)
    p_codes = np.zeros((n, nblk, 32), np.uint8) if want_p else None
    p_meta = np.zeros((n, nblk), np.uint32) if want_p else None
    eps_blk = np.full((n, nblk), np.nan) if want_p else None
    for jb in range(nblk):
        act = np.nonzero(rows >= BLOCK * jb)[0]
        if act.size == 0:
            continue
        keys = np.arange(BLOCK * jb, BLOCK * jb + BLOCK)
        blk = np.full((act.size, BLOCK), -np.inf, s2.dtype)
        nk = min(BLOCK, length - BLOCK * jb)
        blk[:, :nk] = s2[act, BLOCK * jb:BLOCK * jb + nk]
        blk = np.where(keys[None, :] <= rows[act, None], blk, -np.inf).astype(s2.dtype)
        m_new = np.maximum(m[act], blk.max(axis=1))                 # running max
        if exact:
            p = np.exp2(blk - m_new[:, None])
            r = np.exp2(m[act] - m_new)
        else:
            p = exp2_fp16(sub_fp16(blk, m_new[:, None]))            # P16
            r = exp2_fp16(sub_fp16(m[act], m_new)).astype(np.float64)
        p64 = p.astype(np.float64)
        if quantize_p:
            f = hif4.quantize(p64)                                   # P-Reordering
            phat = f["xhat"]
            if want_p:
                c_, m_ = hif4.pack(f)
                p_codes[act, jb] = c_
                p_meta[act, jb] = m_
        else:
            phat = p64
        if want_p:
            with np.errstate(invalid="ignore", divide="ignore"):
                eps_blk[act, jb] = phat.sum(1) / p64.sum(1) - 1.0
        o[act] = o[act] * r[:, None] + phat @ vop[BLOCK * jb:BLOCK * jb + BLOCK]
        l_con[act] = l_con[act] * r + phat.sum(axis=1)                # fused [V|1]
        l_mis[act] = l_mis[act] * r + p64.sum(axis=1)                 # Direct: Z
        m[act] = m_new
    return {"o_num": o, "l_con": l_con, "l_mis": l_mis, "m": m.astype(np.float64),
            "p_codes": p_codes, "p_meta": p_meta, "eps_blk": eps_blk}


def _as_varlen(q, k, v, cu_seqlens):
    if cu_seqlens is None:
        b, s = q.shape[:2]
        return (q.reshape(b * s, *q.shape[2:]), k.reshape(b * s, *k.shape[2:]),
                v.reshape(b * s, *v.shape[2:]), np.arange(b + 1, dtype=np.int64) * s)
    return q, k, v, np.asarray(cu_seqlens, np.int64)


def attention_fwd(q, k, v, s=None, cu_seqlens=None, norm="preorder", operands="hif4",
                  heads=None, seqs=None, rows=None, want_p=False, arith="contract", q_mean=False):
    """HiFA4 forward on fp16 inputs.

    q [B,S,Hq,D] (or [T,Hq,D] with cu_seqlens), k/v [.., Hkv, D], s fp32
    [Hkv, D] or None (no smoothing).  ``heads``/``seqs``/``rows`` restrict the
    computation to a sample (rows are positions within each sequence).
    ``q_mean`` adds the Q-Mean auxiliary (HIF4 operands only).
    ``operands``: "hif4", "fp16" (no quantization, no smoothing) or "p_only"
    (Q, K, V unquantized fp16, no smoothing; only P is HIF4-quantized).
    Returns a dict keyed by (seq, head) with o (float64 O/l), o16, lse, and,
    with want_p, the canonical P^ codes/metadata per (row, block)."""
    qv, kv, vv, cu = _as_varlen(q, k, v, cu_seqlens)
    hq, hkv, d = qv.shape[1], kv.shape[1], qv.shape[2]
    grp = hq // hkv
    if operands == "hif4" and s is not None:
        qv, kv = smooth_apply(qv, kv, s, hkv)
    out = {}
    for b in (range(len(cu) - 1) if seqs is None else seqs):
        t0, t1 = int(cu[b]), int(cu[b + 1])
        length = t1 - t0
        rr = np.arange(length) if rows is None else np.asarray([r for r in rows if r < length])
        vcache = {}
        for h in (range(hq) if heads is None else heads):
            hk = h // grp
            qs, ks, vs = qv[t0:t1, h], kv[t0:t1, hk], vv[t0:t1, hk]
            if arith == "exact":
                q64, k64 = qs.astype(np.float64)[rr], ks.astype(np.float64)
                if q_mean:
                    mu = q64.mean(axis=1)
                    s_raw = (q64 - mu[:, None]) @ k64.T + mu[:, None] * k64.sum(axis=1)[None, :]
                else:
                    s_raw = q64 @ k64.T
                s2 = s_raw * (math.log2(math.e) / math.sqrt(d))
                vop = np.zeros((-(-length // BLOCK) * BLOCK, d)); vop[:length] = vs
                res = online_softmax(s2, vop, rr, length, False, arith="exact")
            elif operands == "hif4":
                corr = None
                if q_mean:
                    mu = token_mean(qs[rr])
                    qf = quantize_rows(zero_mean(qs[rr], mu))
                    corr = (mu, key_sums(ks))
                else:
                    qf = quantize_rows(qs[rr])
                khat = quantize_rows(ks)["xhat"].reshape(length, d)
                if hk not in vcache:
                    vcache[hk] = quantize_tokens(vs)[1]
                s2 = scores_hif4(unit_operands(qf).reshape(len(rr), d), qf["scale"], khat, d, corr)
                res = online_softmax(s2, vcache[hk], rr, length, True, want_p=want_p)
            else:
                # "fp16": the FP16-operand reference; "p_only": the same scores
                # and V with P^ = HIF4(P) as the PV operand (P-only local operator)
                s2 = scores_fp16(qs[rr], ks, d)
                vop = np.zeros((-(-length // BLOCK) * BLOCK, d)); vop[:length] = vs
                res = online_softmax(s2, vop, rr, length, operands == "p_only", want_p=want_p)
            lsum = res["l_mis"] if norm == "inconsistent" else res["l_con"]
            o = res["o_num"] / lsum[:, None]
            res["o"] = o
            res["o16"] = o.astype(np.float32).astype(np.float16)
            res["lse"] = (res["m"] * LN2 + np.log(lsum)).astype(np.float32)
            res["rows"] = rr
            out[(b, h)] = res
    return out


def quantize_qk(q, k, s=None):
    """Smooth-QK then HIF4 of Q~ and K~ along D, in the canonical packed
    layout: codes [..., H, D/64, 32] uint8, meta [..., H, D/64] uint32."""
    hkv = k.shape[-2]
    if s is not None:
        q, k = smooth_apply(q, k, s, hkv)
    qc, qm = hif4.pack(quantize_rows(q))
    kc, km = hif4.pack(quantize_rows(k))
    return qc, qm, kc, km


def quantize_q_mean(q, k, s=None):
    """Q-Mean quantities after Smooth-QK: mu [..., Hq] fp16, kappa [..., Hkv]
    fp32, and HIF4 of Q_z = Q~ - mu in the canonical layout (codes
    [..., Hq, D/64, 32], meta [..., Hq, D/64]).  K^ is that of quantize_qk."""
    hkv = k.shape[-2]
    if s is not None:
        q, k = smooth_apply(q, k, s, hkv)
    mu = token_mean(q)
    qc, qm = hif4.pack(quantize_rows(zero_mean(q, mu)))
    return mu, key_sums(k), qc, qm


def quantize_v(v, cu_seqlens=None):
    """HIF4 of V along tokens, canonical layout per (sequence, kv head,
    channel, 64-token group): codes [G, Hkv, D, 32], meta [G, Hkv, D] where G
    enumerates the token groups of all sequences in order."""
    if cu_seqlens is None:
        b, s = v.shape[:2]
        v = v.reshape(b * s, *v.shape[2:])
        cu = np.arange(b + 1) * s
    else:
        cu = np.asarray(cu_seqlens)
    hkv, d = v.shape[1], v.shape[2]
    codes, metas = [], []
    for b in range(len(cu) - 1):
        for_h_c, for_h_m = [], []
        for h in range(hkv):
            f, _ = quantize_tokens(v[cu[b]:cu[b + 1], h])       # [D, G_b, 64]
            c_, m_ = hif4.pack(f)
            for_h_c.append(c_.transpose(1, 0, 2)); for_h_m.append(m_.T)
        codes.append(np.stack(for_h_c, axis=1)); metas.append(np.stack(for_h_m, axis=1))
    return np.concatenate(codes), np.concatenate(metas)
