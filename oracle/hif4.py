"""HIF4 group quantizer -- the oracle's reading of the format.

Paper: Background, "HIF4" paragraph; Section 4.1; Appendix A (1): a group is
64 contiguous elements with 32 bits of metadata -- a level-1 E6M2 base scale,
8 level-2 one-bit micro-exponents (one per 8 elements), 16 level-3 one-bit
micro-exponents (one per 4 elements) -- and 4-bit sign-magnitude S1P2 elements
(equivalent to E1M2: a 3-bit magnitude code).  Storage is 64*4 + 32 = 288 bits,
4.5 bits per value.

The paper defers the exact conversion to the HIF4 specification, which is not
available; the reading implemented here (all decisions exact, no clipping):

  * element magnitudes are u/4 * s with u in 0..7 (the uniform E1M2 grid);
  * E6M2 is unsigned, bias 31, byte = e<<2 | m, value (1 + m/4) * 2^(e-31);
  * base b = the smallest E6M2 value with 1.75*b >= A, A = group max |x|;
  * level-2 bit j is set iff the 8-element block's max fits the halved range:
    A8[j] <= 0.875*b; a set bit halves the scale of those 8 elements;
  * level-3 bit q is set iff A4[q] <= 0.875*b*2^-E2[q//2]; halves again;
  * element scale s_k = b * 2^-(E2[k//8] + E3[k//4]), step = s_k/4;
  * u_k = floor(|x_k|/step + 1/2)  (round half away from zero);
  * sign bit set iff x_k < 0 and u_k > 0 (zero is stored as +0).

Exactness: every input is an fp16 value (or an fp16 softmax weight), so |x|,
b, step and 1.75*b are exact in float64.  |x|/step is a quotient by (4+m)*2^k;
it is either exactly a half-integer (then float64 division is exact) or at
least 2^-13 relative away from one, far above float64 rounding, so the floor
below is the exact decision.
"""
from __future__ import annotations

import numpy as np

GROUP = 64
E6M2_BIAS = 31


def e6m2_value(byte):
    byte = np.asarray(byte, dtype=np.int64)
    e = byte >> 2
    m = byte & 3
    return (1.0 + m / 4.0) * np.exp2((e - E6M2_BIAS).astype(np.float64))


# All 256 E6M2 values; strictly increasing with the byte.
E6M2_TABLE = e6m2_value(np.arange(256))


def quantize(x):
    """Quantize groups of 64 values along the last axis.

    Returns a dict of exact fields: ``u`` uint8 [...,64] (0..7), ``sign``
    bool [...,64], ``base`` uint8 [...] (E6M2 byte), ``e2`` bool [...,8],
    ``e3`` bool [...,16], and ``xhat`` float64 [...,64] (the dequantized
    values), ``scale`` float64 [...] (the base value b).
    """
    x = np.asarray(x, dtype=np.float64)
    assert x.shape[-1] == GROUP, x.shape
    lead = x.shape[:-1]
    a = np.abs(x)
    A = a.max(-1)
    A8 = a.reshape(*lead, 8, 8).max(-1)
    A4 = a.reshape(*lead, 16, 4).max(-1)
    # level 1: smallest E6M2 value b with 1.75*b >= A (no element can clip)
    base = np.searchsorted(1.75 * E6M2_TABLE, A, side="left")
    if np.any(base > 255):
        raise OverflowError("group maximum exceeds the E6M2 range")
    b = E6M2_TABLE[base]
    # level 2: halve the scale of an 8-block whose max fits in half the range
    e2 = A8 <= 0.875 * b[..., None]
    # level 3: halve again for a 4-block that fits in half of its 8-block range
    e3 = A4 <= 0.875 * b[..., None] * np.exp2(-np.repeat(e2, 2, axis=-1).astype(np.float64))
    shift = np.repeat(e2, 8, axis=-1).astype(np.int64) + np.repeat(e3, 4, axis=-1)
    step = b[..., None] * np.exp2(-shift.astype(np.float64)) / 4.0
    u = np.floor(a / step + 0.5)
    assert np.all(u <= 7)
    sign = (x < 0) & (u > 0)
    xhat = np.where(sign, -u, u) * step
    return {"u": u.astype(np.uint8), "sign": sign, "base": base.astype(np.uint8),
            "e2": e2, "e3": e3, "xhat": xhat, "scale": b}


def dequantize(fields):
    """Rebuild the values from the stored fields alone (codes + metadata)."""
    b = E6M2_TABLE[fields["base"].astype(np.int64)]
    shift = (np.repeat(fields["e2"], 8, axis=-1).astype(np.int64)
             + np.repeat(fields["e3"], 4, axis=-1))
    step = b[..., None] * np.exp2(-shift.astype(np.float64)) / 4.0
    u = fields["u"].astype(np.float64)
    return np.where(fields["sign"], -u, u) * step


def pack(fields):
    """Canonical byte layout: 32 bytes of codes then a 32-bit word of metadata
    per group.  Nibble = sign<<3 | u; element 2i in the low nibble of byte i.
    Metadata word = base | E2 bits << 8 | E3 bits << 16 (bit j = block j)."""
    nib = (fields["sign"].astype(np.uint8) << 3) | fields["u"]
    codes = (nib[..., 0::2] | (nib[..., 1::2] << 4)).astype(np.uint8)
    e2w = (fields["e2"].astype(np.uint32) << np.arange(8, dtype=np.uint32)).sum(-1)
    e3w = (fields["e3"].astype(np.uint32) << np.arange(16, dtype=np.uint32)).sum(-1)
    meta = (fields["base"].astype(np.uint32) | (e2w << 8) | (e3w << 16)).astype(np.uint32)
    return codes, meta


def unpack(codes, meta):
    codes = np.asarray(codes, dtype=np.uint8)
    meta = np.asarray(meta, dtype=np.uint32)
    nib = np.empty(codes.shape[:-1] + (64,), dtype=np.uint8)
    nib[..., 0::2] = codes & 15
    nib[..., 1::2] = codes >> 4
    return {"u": nib & 7, "sign": (nib >> 3).astype(bool),
            "base": (meta & 255).astype(np.uint8),
            "e2": ((meta[..., None] >> (8 + np.arange(8, dtype=np.uint32))) & 1).astype(bool),
            "e3": ((meta[..., None] >> (16 + np.arange(16, dtype=np.uint32))) & 1).astype(bool)}


BITS_PER_GROUP = 64 * 4 + 32     # 288 bits -> 4.5 bits per value
