"""Inputs that drive the running maximum through its special paths: a jump
of more than 25 log2 units in one block (the rescale factor is exactly 0 and
the history is wiped) or a rise over 64 units in steps below 25 (the kernel's
deferred rescale renormalizes).  Integer Q and K keep fp16 scores exact on
the paths whose scores are fp32 sums.  The checks run on the oracle's own
scores, so a case cannot silently miss the path it is meant for."""
import numpy as np

from oracle import attention


def jump_case(kind, lens, hq, hkv, d, seed, jump_block=1):
    """Q in {1, 2}; K in {-1, 0, 1} plus an offset on 5/8 of the channels: 0
    before block `jump_block` and 2 (D=128) or 3 (D=64) from it on ("wipe":
    the scores jump by about 30 log2 units there), or J (D=128) or 1.5 J
    (D=64) on block J up to J = 7 ("renorm": steps of about 15 units).  V
    Gaussian."""
    rng = np.random.default_rng(seed)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    t = int(cu[-1])
    q = rng.integers(1, 3, size=(t, hq, d)).astype(np.float16)
    k = rng.integers(-1, 2, size=(t, hkv, d)).astype(np.float32)
    ch = np.random.default_rng(seed + 1).choice(d, 5 * d // 8, replace=False)
    jump = 2.0 if d == 128 else 3.0
    for b in range(len(lens)):
        pos = np.arange(lens[b])
        blk = np.minimum(pos // 64, 7)
        off = (pos // 64 >= jump_block) * jump if kind == "wipe" else blk * (jump - 1.0) * 0.5 + blk * 0.5
        k[cu[b]:cu[b + 1], :, ch] += off[:, None, None]
    v = rng.standard_normal((t, hkv, d)).astype(np.float32).astype(np.float16)
    return q, k.astype(np.float16), v, cu


def _block_max_steps(s2_rows, L):
    """Per row of a (row, key) fp16 score array: the increases of the running
    maximum from one 64-key block to the next (causal)."""
    steps = []
    for i in range(s2_rows.shape[0]):
        row = s2_rows[i, :i + 1].astype(np.float64)
        bm = [row[64 * J:64 * J + 64].max() for J in range(i // 64 + 1)]
        run = np.maximum.accumulate(bm)
        steps.append(np.diff(run))
    return steps


def _contract_scores(q, k, d, operands):
    if operands == "hif4":
        qf = attention.quantize_rows(q)
        khat = attention.quantize_rows(k)["xhat"].reshape(k.shape[0], d)
        return attention.scores_hif4(attention.unit_operands(qf).reshape(q.shape[0], d), qf["scale"], khat, d)
    return attention.scores_fp16(q, k, d)


def check_jumps(kind, q, k, cu, d, operands, last_row_only=False, min_hits=20):
    """The case really takes the path it is meant for (on the oracle's own
    scores of head 0): a step above 25 (r = 0) on some rows, or, for
    "renorm", every step below 25 and a total rise above 64 on some rows."""
    hit = 0
    for b in range(len(cu) - 1):
        L = cu[b + 1] - cu[b]
        kb = k[cu[b]:cu[b + 1], 0]
        qb = q[cu[b + 1] - 1:cu[b + 1], 0] if last_row_only else q[cu[b]:cu[b + 1], 0]
        s2 = _contract_scores(qb, kb, d, operands)
        if last_row_only:
            bm = [s2[0, 64 * J:64 * J + 64].astype(np.float64).max() for J in range(-(-L // 64))]
            steps = [np.diff(np.maximum.accumulate(bm))]
        else:
            steps = _block_max_steps(s2, L)
        for st in steps:
            if kind == "wipe":
                hit += bool(len(st) and st.max() > 25.5)
            else:
                assert len(st) == 0 or st.max() < 24.5
                hit += bool(len(st) and st.sum() > 66)
    assert hit >= min_hits, (kind, hit)
