"""Decoder of the attention pre-pass's workspace chunks (test code only).

The library's K/V pre-pass writes one chunk per (sequence, kv head, 64-key
block) into the caller's workspace, in the byte layout the attention kernel
streams into LDS.  This module reads those bytes back into element values so
that a test can compare the pre-pass's K^ and V^ with the oracle's element by
element.  The layout is the library's internal one, restated here from its
description (chunk offsets in multiples of 256 bytes, HIF4 chunks padded to
1 KiB):

HIF4 chunk (G = D/64 channel groups):
  * K operand records [2 key halves t][G groups][2 operands]: one record is
    64 lanes x 24 bytes stored as the lanes' first 16 bytes, then their last
    8 bytes; the lane's 192 bits hold 32 FP6 E2M3 fields, field j at bits
    [6j, 6j + 6) (sign = bit 5 of the field).  Lane l holds key 32t + l%32,
    channels 64g + 32(l/32) + j;
  * K scale words [2][G][32 keys]: byte 0 is the E8M0 scale of operand A,
    byte 1 that of operand B (2^(byte - 127)); the element is
    A * 2^(byte0 - 127) + B * 2^(byte1 - 127);
  * V operand records [D/32 channel tiles][2 operands]: lane l holds channel
    32dt + l%32, field s the key 32(s/16) + 8((s%16)/4) + 4(l/32) + s%4;
  * V scale words [D];
  * with Q-Mean, kappa [64 keys] fp32.
FP16 chunk:
  * K [2 key halves][D/16][64 lanes][8 halves]: lane l holds key 32t + l%32,
    channels 16kc + 8(l/32) + e;
  * V [D/32][4 key chunks c = 2t + jp][64 lanes][8 halves]: lane l holds
    channel 32dt + l%32, slot e the key 32t + 8(2jp + e/4) + 4(l/32) + e%4.
"""
import numpy as np

OP_RECORD = 64 * 24


def _ru256(x):
    return (x + 255) & ~255


def hif4_layout(groups, qmean=False):
    k_op = 0
    k_scale = _ru256(2 * groups * 2 * OP_RECORD)
    v_op = k_scale + _ru256(2 * groups * 32 * 4)
    v_scale = v_op + _ru256(2 * groups * 2 * OP_RECORD)
    kappa = v_scale + _ru256(64 * groups * 4)
    end = kappa + (_ru256(64 * 4) if qmean else 0)
    return {"k_op": k_op, "k_scale": k_scale, "v_op": v_op, "v_scale": v_scale, "kappa": kappa,
            "bytes": (end + 1023) & ~1023}


def fp16_layout(d):
    v_op = _ru256(2 * (d // 16) * 64 * 16)
    return {"k_op": 0, "v_op": v_op, "bytes": v_op + _ru256((d // 32) * 4 * 64 * 16)}


def _e2m3_table():
    t = np.zeros(64)
    for f in range(64):
        e, m = (f >> 3) & 3, f & 7
        mag = m / 8.0 if e == 0 else 2.0 ** (e - 1) * (1.0 + m / 8.0)
        t[f] = -mag if f & 32 else mag
    return t


E2M3 = _e2m3_table()


def record_fields(rec):
    """The 32 six-bit fields of each of the 64 lanes of one operand record
    (1536 bytes) -> int64 [64, 32]."""
    rec = np.ascontiguousarray(rec, np.uint8)
    w = np.concatenate([rec[:1024].view(np.uint32).reshape(64, 4),
                        rec[1024:OP_RECORD].view(np.uint32).reshape(64, 2)], axis=1).astype(np.uint64)
    out = np.empty((64, 32), np.int64)
    for j in range(32):
        word, off = divmod(6 * j, 32)
        x = w[:, word] >> np.uint64(off)
        if off > 26:
            x = x | (w[:, word + 1] << np.uint64(32 - off))
        out[:, j] = (x & np.uint64(63)).astype(np.int64)
    return out


def _pair_values(chunk, rec_off, scale_words):
    """Element values A*2^(sa-127) + B*2^(sb-127) of the operand pair at
    rec_off; scale_words [64 lanes] uint32 (the lane's scale word)."""
    fa = record_fields(chunk[rec_off:rec_off + OP_RECORD])
    fb = record_fields(chunk[rec_off + OP_RECORD:rec_off + 2 * OP_RECORD])
    sa = np.exp2((scale_words & 255).astype(np.float64) - 127.0)[:, None]
    sb = np.exp2(((scale_words >> 8) & 255).astype(np.float64) - 127.0)[:, None]
    return E2M3[fa] * sa + E2M3[fb] * sb


def decode_hif4_k(chunk, d):
    """K^ of the chunk's 64 keys -> float64 [64, d]."""
    g_n = d // 64
    lay = hif4_layout(g_n)
    lanes = np.arange(64)
    out = np.full((64, d), np.nan)
    for t in range(2):
        for g in range(g_n):
            so = lay["k_scale"] + (t * g_n + g) * 32 * 4
            words = chunk[so:so + 128].view(np.uint32)[lanes % 32]
            val = _pair_values(chunk, lay["k_op"] + (t * g_n + g) * 2 * OP_RECORD, words)
            keys = 32 * t + lanes % 32
            for j in range(32):
                out[keys, 64 * g + 32 * (lanes // 32) + j] = val[:, j]
    return out


def decode_hif4_v(chunk, d, qmean=False):
    """V^ of the chunk's 64 keys -> float64 [64, d]."""
    lay = hif4_layout(d // 64, qmean)
    lanes = np.arange(64)
    out = np.full((64, d), np.nan)
    vs = chunk[lay["v_scale"]:lay["v_scale"] + 4 * d].view(np.uint32)
    for dt in range(d // 32):
        chan = 32 * dt + lanes % 32
        val = _pair_values(chunk, lay["v_op"] + dt * 2 * OP_RECORD, vs[chan])
        for s in range(32):
            key = 32 * (s // 16) + 8 * ((s % 16) // 4) + 4 * (lanes // 32) + s % 4
            out[key, chan] = val[:, s]
    return out


def decode_hif4_kappa(chunk, d):
    lay = hif4_layout(d // 64, True)
    return chunk[lay["kappa"]:lay["kappa"] + 256].view(np.float32).copy()


def decode_fp16_k(chunk, d):
    kc_n = d // 16
    recs = chunk[:2 * kc_n * 64 * 16].view(np.float16).reshape(2, kc_n, 64, 8)
    out = np.empty((64, d), np.float16)
    lanes = np.arange(64)
    for t in range(2):
        for kc in range(kc_n):
            for e in range(8):
                out[32 * t + lanes % 32, 16 * kc + 8 * (lanes // 32) + e] = recs[t, kc, :, e]
    return out


def decode_fp16_v(chunk, d):
    lay = fp16_layout(d)
    recs = chunk[lay["v_op"]:lay["v_op"] + (d // 32) * 4 * 64 * 16].view(np.float16).reshape(d // 32, 4, 64, 8)
    out = np.empty((64, d), np.float16)
    lanes = np.arange(64)
    for dt in range(d // 32):
        for c in range(4):
            t, jp = c // 2, c % 2
            for e in range(8):
                key = 32 * t + 8 * (2 * jp + e // 4) + 4 * (lanes // 32) + e % 4
                out[key, 32 * dt + lanes % 32] = recs[dt, c, :, e]
    return out
