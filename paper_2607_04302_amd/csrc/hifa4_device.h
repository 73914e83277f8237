// Device-side building blocks shared by the HiFA4 kernels (gfx950).
//
// HIF4 group quantization (paper, Background "HIF4" paragraph; Section 4.1)
// under the library's reading: unsigned E6M2 base b = smallest value with
// 1.75*b >= max|x| (bias 31); level-2 (8 elements) and level-3 (4 elements)
// one-bit micro-exponents that halve the scale when the block's maximum fits
// in half of the range; element code u = round-half-away(|x| / step),
// step = b * 2^-(E2+E3) / 4.
//
// MFMA operand encoding.  A HIF4 element equals o * b/4 with o = u * 2^-sh,
// u in 0..7 and sh = E2+E3 in 0..2.  Every such o is exactly representable in
// the OCP FP6 E2M3 format (values m/8 and (1+m/8)*2^(e-1)), which E2M1 (FP4)
// cannot hold (5 and 7 need three significant bits).  The kernels therefore
// feed o as FP6 E2M3 to the block-scaled F8F6F4 MFMA (same issue rate as
// FP4) with unit E8M0 scales, so every group dot product sum(o_q * o_k) is
// exact in the fp32 accumulator, and apply the E6M2 bases (which carry two
// mantissa bits that an E8M0 scale cannot) in an fp32 epilogue.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hifa4 {

typedef _Float16 half_t;
typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef _Float16 h32_t __attribute__((ext_vector_type(32)));
typedef float f16v_t __attribute__((ext_vector_type(16)));
typedef int i6_t __attribute__((ext_vector_type(6)));
typedef int i8_t __attribute__((ext_vector_type(8)));

// FP6 E2M3 encoding of 1.0 (sign 0, exponent 01, mantissa 000), replicated
// in 6-bit fields: the all-ones operand of the fused normalizer [V^ | 1].
constexpr uint32_t kE2M3One = 0x08;


// Smallest E6M2 byte whose value b satisfies 1.75*b >= A (A >= 0, an fp16 or
// fp16-softmax value held exactly in fp32), without branches.  Write
// A = s*2^E with s in [1,2).  The values 1.75*b of the bases near A are
// 1.09375, 1.3125, 1.53125 (mantissas m = 1, 2, 3, exponent E-1), 1.75 and
// 2.1875 (m = 0, 1, exponent E) times 2^E, so the smallest covering base is
// code 4(E+30) + 1 + [s > 1.09375] + [s > 1.3125] + [s > 1.53125] + [s > 1.75];
// the comparisons are exact on the fp32 significand bits.  A = 0 gives 0.
__device__ __forceinline__ uint32_t e6m2_ceil(float A) {
  const uint32_t bits = __float_as_uint(A);
  const uint32_t mant = bits & 0x7FFFFFu;
  const int c = (int)(mant > 0xC0000u) + (int)(mant > 0x280000u) + (int)(mant > 0x440000u) +
                (int)(mant > 0x600000u);
  const int code = 4 * (int)(bits >> 23) - 387 + c;
  return A > 0.0f ? (uint32_t)code : 0u;
}

// E6M2 value b = (1 + m/4) * 2^(e-31) of byte e<<2|m, built from its bits.
__device__ __forceinline__ float e6m2_bits_value(uint32_t code) {
  return __uint_as_float((code << 21) + 0x30000000u);
}

// R = (4/b) * (1 + 2^-18), rounded: for the 4 base mantissas the constant
// fp32(16/(4+m) * (1 + 2^-18)), then an exact power-of-two scaling by
// 2^(31-e) applied to the exponent field.
//
// Element rounding uses o = fl(a*R + C_sh) - C_sh with C_sh = 1.5*2^(23-sh)
// (fp32) or 1.5*2^(10-sh) (fp16 destination): the fused multiply-add rounds
// the exact product a*R once onto the grid 2^-sh, which is u*2^-sh with
// u = round-half-to-even(a/step * (1+beta)).  a/step is an fp16 value divided
// by (4+m)*2^k: a non-tie lies at least 2^-12 (relative) from a half-integer
// while beta ~ 2^-18, so those round as exactly as without beta; an exact tie
// n+1/2 is pushed strictly above and rounds away from zero.  The result is
// exactly round-half-away(a/step).
__device__ __forceinline__ float hif4_rcp_step(uint32_t code) {
  const uint32_t m = code & 3u;
  const uint32_t lo = (m & 1u) ? 0x404ccd00u : 0x40800020u;   // m = 1 : 0
  const uint32_t hi = (m & 1u) ? 0x40124949u : 0x402aaad5u;   // m = 3 : 2
  const uint32_t cb = (m & 2u) ? hi : lo;
  return __uint_as_float(cb + (uint32_t)((31 - (int)(code >> 2)) << 23));
}

// E6M2 value of a base byte: (1 + m/4) * 2^(e - 31).
__device__ __forceinline__ float e6m2_value(uint32_t code) { return e6m2_bits_value(code); }

__device__ __forceinline__ float round_const(int sh) {
  return sh == 0 ? 12582912.0f : (sh == 1 ? 6291456.0f : 3145728.0f);
}

// o = u * 2^-sh for one element magnitude a (>= 0).
__device__ __forceinline__ float hif4_elem(float a, float R, float C) {
  return __builtin_fmaf(a, R, C) - C;
}

// fp16 softmax exponential E(x) = fp16(2^x) for a pair of fp16 x (x = -inf
// gives 0): v_exp_f16 on the low half, then its SDWA form on the high half,
// which keeps the low half of the destination.  The SDWA form reads the
// destination to preserve it, so it must wait for the transcendental result
// (the s_nop; the compiler does not see this dependency inside the asm).
// On gfx950 v_exp_f16 returns the correctly rounded value for every fp16
// input x <= 0 (checked exhaustively; the library's exp2 self-test entry
// point re-checks this routine on the device).
__device__ __forceinline__ h2_t exp2_h2(h2_t x) {
  h2_t y;
  asm("v_exp_f16 %0, %1\n\ts_nop 1\n\tv_exp_f16_sdwa %0, %1 dst_sel:WORD_1 dst_unused:UNUSED_PRESERVE src0_sel:WORD_1"
      : "=&v"(y)
      : "v"(x));
  return y;
}

// fp16(a*b) for fp32 a and b, the exact product rounded once (v_fma_mix with
// an fp16 destination rounds the fused result once; low half of the result).
__device__ __forceinline__ half_t mul_rn16(float a, float b) {
  half_t y;
  asm("v_fma_mixlo_f16 %0, %1, %2, 0" : "=v"(y) : "v"(a), "v"(b));
  return y;
}

// Pack fp16(fp32(a*c)) and fp16(fp32(b*c)): the products are rounded to fp32,
// then converted to fp16 (round to nearest even) by one packed conversion.
__device__ __forceinline__ h2_t scale2_to_f16(float a, float b, float c) {
  const float ya = a * c, yb = b * c;
  h2_t y;
  asm("v_cvt_pk_f16_f32 %0, %1, %2" : "=v"(y) : "v"(ya), "v"(yb));
  return y;
}

// Pack fp16(a) and fp16(b) (round to nearest even) into one register.
__device__ __forceinline__ h2_t pack2_f16(float a, float b) {
  h2_t y;
  asm("v_cvt_pk_f16_f32 %0, %1, %2" : "=v"(y) : "v"(a), "v"(b));
  return y;
}

// Pack fp16(a*c) and fp16(b*c) (each rounded once) into one register.
__device__ __forceinline__ h2_t mul2_rn16(float a, float b, float c) {
  h2_t y;
  asm("v_fma_mixlo_f16 %0, %1, %3, 0\n\tv_fma_mixhi_f16 %0, %2, %3, 0" : "=&v"(y) : "v"(a), "v"(b), "v"(c));
  return y;
}

// fp16 nearest to the exact quotient k/s (k an fp16 value, s > 0 fp32): the
// correctly rounded fp32 quotient rounds to the same fp16 unless it sits
// exactly on an fp16 midpoint; there the exact remainder k - q*s (exact in
// fp32 for a correctly rounded q) tells on which side the true quotient lies.
__device__ __forceinline__ half_t div_rn16(float k, float s) {
  const float q = k / s;
  const half_t h = (half_t)q;
  const float hv = (float)h;
  if (hv == q) return h;
  const uint16_t hb = __builtin_bit_cast(uint16_t, h);
  // neighbour of h on q's side (magnitude up if |q| > |h|)
  const uint16_t nbb = (fabsf(q) > fabsf(hv)) ? (uint16_t)(hb + 1) : (uint16_t)(hb - 1);
  const half_t nb = __builtin_bit_cast(half_t, nbb);
  const float mid = 0.5f * (hv + (float)nb);
  if (q != mid) return h;
  const float r = __builtin_fmaf(-q, s, k);        // exact remainder
  if (r == 0.0f) return h;                          // exact tie: h is the even one
  const bool above = r > 0.0f;                      // true quotient > q (s > 0)
  const bool nb_above = (float)nb > q;
  return (above == nb_above) ? nb : h;
}

// The same quotient from a reciprocal rs = RN32(1/s): k*rs = (k/s)(1 + d)
// with |d| <= 2^-24, so q = RN32(k*rs) lies within 1.5 fp32 ulps of k/s and
// RN16(q) = RN16(k/s) unless q's bits below the fp16 precision (the low 13
// mantissa bits) are within 3 of the halfway pattern 0x1000, or q is in
// fp16's subnormal range; those take div_rn16.
__device__ __forceinline__ half_t div_rn16_rcp(float k, float s, float rs) {
  const float q = k * rs;
  const uint32_t b = __float_as_uint(q);
  const bool near_mid = ((b & 0x1FFFu) - 0xFFDu) < 7u;
  const bool tiny = (b & 0x7F800000u) < 0x38800000u && (b & 0x7FFFFFFFu) != 0u;
  if (__builtin_expect(near_mid || tiny, 0)) return div_rn16(k, s);
  return (half_t)q;
}

__device__ __forceinline__ float shfl_xor32(float v) {
  return __shfl_xor(v, 32);
}
__device__ __forceinline__ uint32_t shfl_xor32_u(uint32_t v) {
  return (uint32_t)__shfl_xor((int)v, 32);
}

// ---------------------------------------------------------------------------
// Lane-split group quantization.  A 64-element group is held by a lane pair
// (lane l and l^32), 32 elements each, as 8 complete 4-element blocks.
// `q4[k]` is the global index (0..15) of the lane's k-th 4-block, and a4[k]
// its maximum magnitude.  Both lanes compute identical group metadata.
struct GroupMeta {
  uint32_t base;    // E6M2 byte
  uint32_t e2;      // 8 bits
  uint32_t e3;      // 16 bits
  float b;          // base value
};

// a4_all[0..15]: the maxima of all 16 4-blocks of the group, in block order.
__device__ __forceinline__ GroupMeta group_meta(const float a4_all[16]) {
  GroupMeta g;
  float A8[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) A8[j] = fmaxf(a4_all[2 * j], a4_all[2 * j + 1]);
  float A = A8[0];
#pragma unroll
  for (int j = 1; j < 8; ++j) A = fmaxf(A, A8[j]);
  g.base = e6m2_ceil(A);
  g.b = e6m2_value(g.base);
  const float half_range = 0.875f * g.b;
  g.e2 = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) g.e2 |= (A8[j] <= half_range ? 1u : 0u) << j;
  g.e3 = 0;
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    const float lim = ((g.e2 >> (q >> 1)) & 1u) ? 0.5f * half_range : half_range;
    g.e3 |= (a4_all[q] <= lim ? 1u : 0u) << q;
  }
  return g;
}

__device__ __forceinline__ int block_shift(const GroupMeta& g, int q4) {
  return (int)((g.e2 >> (q4 >> 1)) & 1u) + (int)((g.e3 >> q4) & 1u);
}

// Which 4-blocks a lane holds.  kRows: lane half h holds the contiguous
// elements [32h, 32h+32), i.e. blocks 8h..8h+7 (Q, K along channels).
// kKeys: the lane's k-th block is (t = k/4, j = k%4), elements
// 32t + 8j + 4h + [0,4), i.e. block 8t + 2j + h (V along tokens, and P,
// following the 32x32 MFMA output layout of S^T).
enum { kRows = 0, kKeys = 1 };

template <int LAYOUT>
__device__ __forceinline__ int own_block(int k, int h) {
  return LAYOUT == kRows ? 8 * h + k : 8 * (k >> 2) + 2 * (k & 3) + h;
}

// Assemble the 16 block maxima of the group from the lane's 8 and its
// partner's (lane l^32) 8, with static register indexing.
template <int LAYOUT>
__device__ __forceinline__ void gather_a4(const float own[8], float all[16], int h) {
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const float other = shfl_xor32(own[k]);
    const int lo = LAYOUT == kRows ? k : 8 * (k >> 2) + 2 * (k & 3);
    const int hi = LAYOUT == kRows ? 8 + k : lo + 1;
    all[lo] = h ? other : own[k];
    all[hi] = h ? own[k] : other;
  }
}

}  // namespace hifa4
