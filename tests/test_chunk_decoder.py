"""CPU pins of the chunk decoder used by the pre-pass GPU tests: the FP6 E2M3
value table, the 6-bit field packing of an operand record (built here from a
Python integer per lane, independently of the decoder's word arithmetic) and
the two-operand element value with its E8M0 scales."""
import numpy as np

from _chunks import E2M3, OP_RECORD, _pair_values, record_fields


def test_e2m3_values():
    # sign | exponent (2 bits, bias 1) | mantissa (3 bits); E = 0 is subnormal
    assert E2M3[0b000000] == 0.0
    assert E2M3[0b000001] == 0.125
    assert E2M3[0b000111] == 0.875
    assert E2M3[0b001000] == 1.0
    assert E2M3[0b010100] == 3.0
    assert E2M3[0b011111] == 7.5
    assert E2M3[0b111111] == -7.5
    assert E2M3[0b100000] == 0.0 and np.signbit(E2M3[0b100000])
    # the u * 2^-sh values of HIF4 elements (u <= 7, sh <= 2) are all present
    want = {u * 2.0 ** -sh for u in range(8) for sh in range(3)}
    assert want <= set(E2M3.tolist())


def _record_from_fields(fields):
    rec = np.zeros(OP_RECORD, np.uint8)
    for lane in range(64):
        v = 0
        for j in range(32):
            v |= int(fields[lane, j]) << (6 * j)
        lo = (v & ((1 << 128) - 1)).to_bytes(16, "little")
        hi = (v >> 128).to_bytes(8, "little")
        rec[16 * lane:16 * lane + 16] = np.frombuffer(lo, np.uint8)
        rec[1024 + 8 * lane:1024 + 8 * lane + 8] = np.frombuffer(hi, np.uint8)
    return rec


def test_record_fields_roundtrip():
    rng = np.random.default_rng(0)
    f = rng.integers(0, 64, (64, 32))
    assert np.array_equal(record_fields(_record_from_fields(f)), f)


def test_pair_value_applies_both_scales():
    fa = np.zeros((64, 32), np.int64)
    fb = np.zeros((64, 32), np.int64)
    fa[:, 0] = 0b010100          # 3.0
    fb[:, 0] = 0b110100          # -3.0
    fa[:, 1] = 0b000010          # 0.25
    chunk = np.concatenate([_record_from_fields(fa), _record_from_fields(fb)])
    # scale bytes: A 2^-33 (94), B 2^-35 (92): 1.75 * 2^-33 per unit code
    words = np.full(64, 94 | (92 << 8), np.uint32)
    val = _pair_values(chunk, 0, words)
    assert np.all(val[:, 0] == 3.0 * 2.0 ** -33 - 3.0 * 2.0 ** -35)
    assert np.all(val[:, 1] == 0.25 * 2.0 ** -33)
    assert np.all(val[:, 2:] == 0.0)
