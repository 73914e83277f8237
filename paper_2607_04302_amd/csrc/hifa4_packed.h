// Packed-fp16 building blocks of the HIF4 quantizers (gfx950), shared by the
// attention kernels and the K/V pre-pass.
//
// HIF4 group quantization under the library's reading (the paper's HIF4
// paragraph in Background; Section 4.1): E6M2 base b = the smallest value with
// 1.75 b >= max|x|, level-2 and level-3 micro-exponents that halve the scale
// of 8- and 4-element blocks whose maximum fits in half of the range, element
// code u = round-half-away(|x| / step).  A group of 64 is held by a lane
// pair (l, l^32), 32 elements each as 16 packed fp16 pairs; every decision is
// taken on exact fp16 values: maxima with packed fp16 max, the base from the
// fp32 bits of the maximum, the shift of each 4-block by saturating 16-bit
// arithmetic on the bit patterns, and each magnitude rounded onto its grid by
// one mixed-precision fused multiply-add.
#pragma once

#include "hifa4_device.h"

namespace hifa4 {

// Lane-pair exchange with v_permlane32_swap(v, v): it swaps the upper 32
// lanes of the first copy with the lower 32 lanes of the second, so lanes
// 0..31 see (own, partner) and lanes 32..63 see (partner, own).  Symmetric
// combinations need no select.
struct Pair32 {
  uint32_t x, y;
};
__device__ __forceinline__ Pair32 pair32(uint32_t v) {
  const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return Pair32{r[0], r[1]};
}
__device__ __forceinline__ h2_t max_with_partner(h2_t v) {
  const Pair32 p = pair32(__builtin_bit_cast(uint32_t, v));
  h2_t y;
  asm("v_pk_max_f16 %0, %1, %2" : "=v"(y) : "v"(p.x), "v"(p.y));
  return y;
}
__device__ __forceinline__ float add_with_partner(float v) {
  const Pair32 p = pair32(__builtin_bit_cast(uint32_t, v));
  return __builtin_bit_cast(float, p.x) + __builtin_bit_cast(float, p.y);
}
// The partner lane's value (h = lane / 32).
__device__ __forceinline__ h2_t partner_h2(h2_t v, int h) {
  const Pair32 p = pair32(__builtin_bit_cast(uint32_t, v));
  return __builtin_bit_cast(h2_t, h ? p.x : p.y);
}

// o = fp16(p*R + C) - C for both halves of p (fp16), R fp32 and C half SEL
// of cp (fp16).  The fused value is rounded once to fp16, onto the grid of C;
// the subtraction is exact.
template <int SEL>
__device__ __forceinline__ h2_t grid_round2(h2_t p, float R, h2_t cp) {
  h2_t y;
  if (SEL == 0)
    asm("v_fma_mixlo_f16 %0, %1, %2, %3 op_sel:[0,0,0] op_sel_hi:[1,0,1]\n\t"
        "v_fma_mixhi_f16 %0, %1, %2, %3 op_sel:[1,0,0] op_sel_hi:[1,0,1]\n\t"
        "v_pk_add_f16 %0, %0, %3 op_sel:[0,0] op_sel_hi:[1,0] neg_lo:[0,1] neg_hi:[0,1]"
        : "=&v"(y)
        : "v"(p), "v"(R), "v"(cp));
  else
    asm("v_fma_mixlo_f16 %0, %1, %2, %3 op_sel:[0,0,1] op_sel_hi:[1,0,1]\n\t"
        "v_fma_mixhi_f16 %0, %1, %2, %3 op_sel:[1,0,1] op_sel_hi:[1,0,1]\n\t"
        "v_pk_add_f16 %0, %0, %3 op_sel:[0,1] op_sel_hi:[1,1] neg_lo:[0,1] neg_hi:[0,1]"
        : "=&v"(y)
        : "v"(p), "v"(R), "v"(cp));
  return y;
}

// Rounding constants of a pair of 4-blocks (low / high half): with A4 the
// 4-block maximum, A8 its 8-block maximum and h, q the fp16 floors of 0.875b
// and 0.4375b, the block's shift is sh = [A8 <= h] + [A4 <= (A8 <= h ? q : h)]
// = 2 - n with n = [A4 > h] + ([A8 > h] | [A4 > q]), and its constant
// 1.5 * 2^(10 - sh) has the fp16 bits 0x5E00 + n * 0x400.  Non-negative fp16
// values order like their bit patterns, so each test is a saturating 16-bit
// subtraction clamped to 1.
__device__ __forceinline__ h2_t grid_consts(h2_t a4, h2_t a8, h2_t th_h, h2_t th_q, uint32_t k400, uint32_t k5e00) {
  h2_t n;
  uint32_t t, w;
  asm("v_pk_sub_u16 %0, %3, %5 clamp\n\t"       // n = sat(A4 - h)
      "v_pk_sub_u16 %1, %4, %5 clamp\n\t"       // t = sat(A8 - h)
      "v_pk_sub_u16 %2, %3, %6 clamp\n\t"       // w = sat(A4 - q)
      "v_pk_max_u16 %1, %1, %2\n\t"
      "v_pk_min_u16 %0, %0, 1 op_sel_hi:[1,0]\n\t"
      "v_pk_min_u16 %1, %1, 1 op_sel_hi:[1,0]\n\t"
      "v_pk_add_u16 %0, %0, %1\n\t"
      "v_pk_mad_u16 %0, %0, %7, %8"
      : "=&v"(n), "=&v"(t), "=&v"(w)
      : "v"(a4), "v"(a8), "v"(th_h), "v"(th_q), "v"(k400), "v"(k5e00));
  return n;
}

// Packed fp16 max.  Written as an instruction so that the compiler does not
// canonicalize its (finite or -inf, never NaN) operands first.
__device__ __forceinline__ h2_t hmax2(h2_t a, h2_t b) {
  h2_t y;
  asm("v_pk_max_f16 %0, %1, %2" : "=v"(y) : "v"(a), "v"(b));
  return y;
}
// max of the two halves, in both halves
__device__ __forceinline__ h2_t hmax_halves(h2_t a) {
  h2_t y;
  asm("v_pk_max_f16 %0, %1, %1 op_sel:[0,1] op_sel_hi:[1,0]" : "=v"(y) : "v"(a));
  return y;
}
// max(a.lo, a.hi) in the low half and max(b.lo, b.hi) in the high half
// (two SDWA maxima in one block).
__device__ __forceinline__ h2_t hmax_pairs(h2_t a, h2_t b) {
  h2_t y;
  asm("v_max_f16_sdwa %0, %1, %1 dst_sel:WORD_0 dst_unused:UNUSED_PAD src0_sel:WORD_0 src1_sel:WORD_1\n\t"
      "v_max_f16_sdwa %0, %2, %2 dst_sel:WORD_1 dst_unused:UNUSED_PRESERVE src0_sel:WORD_0 src1_sel:WORD_1"
      : "=&v"(y)
      : "v"(a), "v"(b));
  return y;
}

// The value of lane l^32 through the LDS crossbar (ds_bpermute; `addr` is
// 4 * (l ^ 32)).  Used where several exchanges are independent so that their
// latency overlaps and the VALU stays free.
__device__ __forceinline__ uint32_t partner_bperm(uint32_t v, int addr) {
  return (uint32_t)__builtin_amdgcn_ds_bpermute(addr, (int)v);
}

// fp16(x * s) for both halves of x with per-half fp32 scales: the exact
// product rounded once (v_fma_mix with an fp16 destination).
__device__ __forceinline__ h2_t smooth_mul2(h2_t x, float s0, float s1) {
  h2_t y;
  asm("v_fma_mixlo_f16 %0, %1, %2, 0 op_sel:[0,0,0] op_sel_hi:[1,0,0]\n\t"
      "v_fma_mixhi_f16 %0, %1, %3, 0 op_sel:[1,0,0] op_sel_hi:[1,0,0]"
      : "=&v"(y)
      : "v"(x), "v"(s0), "v"(s1));
  return y;
}

// |x| for both halves (max(x, -x); the values are finite).
__device__ __forceinline__ h2_t habs2(h2_t x) {
  h2_t y;
  asm("v_pk_max_f16 %0, %1, %1 neg_lo:[0,1] neg_hi:[0,1]" : "=v"(y) : "v"(x));
  return y;
}

// max(a, b) for both halves, written as an instruction (no canonicalization).
__device__ __forceinline__ h2_t hmax2_q(h2_t a, h2_t b) {
  h2_t y;
  asm("v_pk_max_f16 %0, %1, %2" : "=v"(y) : "v"(a), "v"(b));
  return y;
}

// fp16 nearest to a float64 value (ties to even), rounded once: the value is
// first rounded to odd in fp32 (which keeps 13 more significand bits than
// fp16, enough for the second rounding to be exact), then to fp16.
__device__ __forceinline__ half_t rn16_from_f64(double x) {
  const float f = (float)x;
  uint32_t b = __float_as_uint(f);
  const double fd = (double)f;
  if (fd != x) {
    if (fabs(fd) > fabs(x)) b -= 1u;      // one fp32 step toward zero
    b |= 1u;                             // sticky bit: round to odd
  }
  return (half_t)__uint_as_float(b);
}

// P^ = HIF4(P) of one 64-key block held in the S^T accumulator layout (lane
// half h holds keys 32t + 8j + 4h + [0,4) of 4-block (t, j) in the packed
// registers p2[t][2j], p2[t][2j+1]; the 8-blocks pair with lane l^32).  A is
// the block maximum (an fp16 value).  Returns the operand values
// o = u * 2^-sh in the order of the packed registers (slot 16t + 2v2 + e =
// half e of p2[t][v2]) and the E6M2 base.  With DEBUG, a non-null dcodes /
// dmeta receive the lane's share of the canonical codes and the metadata
// word.
struct PQuant {
  h32_t ov;
  uint32_t base;
  float bval;
};

template <bool DEBUG>
__device__ __forceinline__ PQuant quantize_p_block(const h2_t (&p2)[2][8], float A, int lane, int h, uint8_t* dcodes,
                                                   uint32_t* dmeta) {
  PQuant out;
  // Maxima are packed in pairs of 4-blocks: a4[t][jp] = (A4(t, 2jp), A4(t, 2jp+1)).
  const uint32_t base = e6m2_ceil(A);
  const float bval = e6m2_value(base);
  const float R = hif4_rcp_step(base);
  // fp16 floors of the half and quarter ranges: an fp16 value x satisfies
  // x <= 0.875b iff x <= floor16(0.875b) (round-toward-zero conversion).
  const h2_t thr = __builtin_bit_cast(h2_t, __builtin_amdgcn_cvt_pkrtz(0.875f * bval, 0.4375f * bval));
  const h2_t th_h = {thr[0], thr[0]}, th_q = {thr[1], thr[1]};
  const uint32_t k400 = 0x04000400u, k5e00 = 0x5E005E00u;
  h2_t cst[2][2];       // rounding constants of 4-blocks (t, 2jp), (t, 2jp+1)
  h2_t a4s[2][2], a4p[2][2];
  uint32_t e2bits = 0, e3bits = 0;
  const int paddr = 4 * (lane ^ 32);
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int jp = 0; jp < 2; ++jp) {
      const h2_t m0 = hmax2(p2[t][4 * jp], p2[t][4 * jp + 1]);       // 4-block 2jp, two partial maxima
      const h2_t m1 = hmax2(p2[t][4 * jp + 2], p2[t][4 * jp + 3]);   // 4-block 2jp+1
      a4s[t][jp] = hmax_pairs(m0, m1);
      a4p[t][jp] = __builtin_bit_cast(h2_t, partner_bperm(__builtin_bit_cast(uint32_t, a4s[t][jp]), paddr));
    }
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int jp = 0; jp < 2; ++jp) {
      const h2_t a4 = a4s[t][jp];
      const h2_t a8 = hmax2(a4, a4p[t][jp]);
      cst[t][jp] = grid_consts(a4, a8, th_h, th_q, k400, k5e00);
      if (DEBUG) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const int j = 2 * jp + e;
          const bool e2 = a8[e] <= th_h[e];
          const bool e3 = a4[e] <= (e2 ? th_q[e] : th_h[e]);
          e2bits |= (uint32_t)e2 << (4 * t + j);
          e3bits |= (uint32_t)e3 << (8 * t + 2 * j + h);
          const bool e3o = a4p[t][jp][e] <= (e2 ? th_q[e] : th_h[e]);
          e3bits |= (uint32_t)e3o << (8 * t + 2 * j + (h ^ 1));
        }
      }
    }
  // o = u * 2^-sh: one fp16 fma rounds P*R onto the grid 2^-sh, a packed
  // subtraction removes the offset (both exact).
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int v2 = 0; v2 < 8; ++v2) {
      // 4-block j = v2/2 of tile t: its constant is half (j & 1) of cst[t][j >> 1]
      const h2_t cp = cst[t][v2 >> 2];
      const h2_t tt = ((v2 >> 1) & 1) ? grid_round2<1>(p2[t][v2], R, cp) : grid_round2<0>(p2[t][v2], R, cp);
      out.ov[16 * t + 2 * v2] = tt[0];
      out.ov[16 * t + 2 * v2 + 1] = tt[1];
    }
  if (DEBUG && dcodes) {
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int q4 = 8 * t + 2 * j + h;
        const int sh = (int)((e2bits >> (4 * t + j)) & 1u) + (int)((e3bits >> q4) & 1u);
        uint32_t nib[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) nib[i] = (uint32_t)((float)out.ov[16 * t + 4 * j + i] * (float)(1 << sh));
        dcodes[16 * t + 4 * j + 2 * h] = (uint8_t)(nib[0] | (nib[1] << 4));
        dcodes[16 * t + 4 * j + 2 * h + 1] = (uint8_t)(nib[2] | (nib[3] << 4));
      }
    if (h == 0) *dmeta = base | (e2bits << 8) | (e3bits << 16);
  }
  out.base = base;
  out.bval = bval;
  return out;
}

// The quantizer's output for one lane: its 32 FP6 E2M3 fields, the group's
// E6M2 base byte and base value.
struct GroupOps {
  i6_t pk;
  uint32_t base;
  float bval;
};

// HIF4 of a group in row layout: lane half h holds elements 32h..32h+31 as
// x[i] = (element 32h+2i, 32h+2i+1), i.e. 4-blocks 8h..8h+7 and 8-blocks
// 4h..4h+3, so only the group maximum needs the partner lane.  FP6 slot s =
// element 32h + s, value +-u*2^-sh (a negative value whose code is 0 becomes
// -0, which the MFMA treats as 0).  Used for Q and K along the head dimension.
__device__ __forceinline__ GroupOps rows_quantize(const h2_t (&x)[16]) {
  h2_t ax[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) ax[i] = habs2(x[i]);
  // 4-block k = pairs 2k, 2k+1; a4p[j] = (A4[2j], A4[2j+1]) = 8-block j's halves
  h2_t a4p[4], a8[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const h2_t m0 = hmax2_q(ax[4 * j], ax[4 * j + 1]);
    const h2_t m1 = hmax2_q(ax[4 * j + 2], ax[4 * j + 3]);
    a4p[j] = hmax_pairs(m0, m1);
    a8[j] = hmax_halves(a4p[j]);
  }
  const h2_t lane_max = hmax2_q(hmax2_q(a8[0], a8[1]), hmax2_q(a8[2], a8[3]));
  const h2_t gmax = max_with_partner(lane_max);
  const float A = (float)gmax[0];
  GroupOps r;
  r.base = e6m2_ceil(A);
  r.bval = e6m2_value(r.base);
  const float R = hif4_rcp_step(r.base);
  const h2_t thr = __builtin_bit_cast(h2_t, __builtin_amdgcn_cvt_pkrtz(0.875f * r.bval, 0.4375f * r.bval));
  const h2_t th_h = {thr[0], thr[0]}, th_q = {thr[1], thr[1]};
  const uint32_t k400 = 0x04000400u, k5e00 = 0x5E005E00u;
  h32_t ov;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const h2_t cst = grid_consts(a4p[j], a8[j], th_h, th_q, k400, k5e00);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int i = 4 * j + e;                 // pair i belongs to 4-block 2j + e/2
      const h2_t o = (e >> 1) ? grid_round2<1>(ax[i], R, cst) : grid_round2<0>(ax[i], R, cst);
      const uint32_t sgn = __builtin_bit_cast(uint32_t, x[i]) & 0x80008000u;
      const h2_t os = __builtin_bit_cast(h2_t, __builtin_bit_cast(uint32_t, o) | sgn);
      ov[2 * i] = os[0];
      ov[2 * i + 1] = os[1];
    }
  }
  r.pk = __builtin_amdgcn_cvt_scalef32_pk32_fp6_f16(ov, 1.0f);
  return r;
}

// HIF4 of a signed group in key layout (that of P^ in the S^T accumulator:
// x[t][v2] holds elements 32t + 8(v2/2) + 4h + 2(v2%2) + {0, 1}; 8-blocks pair
// with lane l^32).  FP6 slot 16t + 2v2 + e = half e of x[t][v2].  Used for V
// along tokens.
__device__ __forceinline__ GroupOps keys_quantize(const h2_t (&x)[2][8], int lane, int h) {
  h2_t ax[2][8];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int v2 = 0; v2 < 8; ++v2) ax[t][v2] = habs2(x[t][v2]);
  h2_t m = ax[0][0];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int v2 = 0; v2 < 8; ++v2)
      if (t > 0 || v2 > 0) m = hmax2_q(m, ax[t][v2]);
  const h2_t gmax = hmax_halves(max_with_partner(m));
  const PQuant pq = quantize_p_block<false>(ax, (float)gmax[0], lane, h, nullptr, nullptr);
  h32_t ov;
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int v2 = 0; v2 < 8; ++v2) {
      const h2_t o = {pq.ov[16 * t + 2 * v2], pq.ov[16 * t + 2 * v2 + 1]};
      const uint32_t sgn = __builtin_bit_cast(uint32_t, x[t][v2]) & 0x80008000u;
      const h2_t os = __builtin_bit_cast(h2_t, __builtin_bit_cast(uint32_t, o) | sgn);
      ov[16 * t + 2 * v2] = os[0];
      ov[16 * t + 2 * v2 + 1] = os[1];
    }
  GroupOps r;
  r.pk = __builtin_amdgcn_cvt_scalef32_pk32_fp6_f16(ov, 1.0f);
  r.base = pq.base;
  r.bval = pq.bval;
  return r;
}

}  // namespace hifa4
