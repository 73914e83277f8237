// HiFA4 causal prefill attention forward (gfx950).
//
// Paper: Algorithm 1 (C4V16 without Q-Mean); Background, "FlashAttention
// tiling"; Section 4.5 (P-Reordering, fused normalizer P^[V^|1]); "P-Reordering
// under online softmax"; Appendix C (FP16 state, GQA).
//
// Work decomposition.  A workgroup of 4 waves owns one KV head, one sequence
// and a tile of queries: 4 query heads x 32 rows when the GQA group has >= 4
// heads, 2 heads x 64 rows for groups of 2, one head x 128 rows otherwise, so
// every K/V block staged in LDS serves 4 waves.  Each wave holds 32 query rows
// of one head.  Workgroups are issued longest-first (causal tiles with more
// key blocks first).
//
// Per 64-key block (one P group, one V group) and wave:
//   S^T[key, q] = K^ Q^T with two 32x32x64 FP6 MFMAs per 64-channel group
//     (the A operand is the pre-pass K tile in LDS, B the Q tile quantized in
//     registers at kernel start); each MFMA sum is exact, the fp32 epilogue
//     applies b_Q*b_K per group and sums the groups in order, then x c and to
//     fp16.  In S^T each lane holds one query and 32 of the block's keys, so
//     row maxima are in-lane plus one exchange with lane l^32;
//   FP16 softmax: m_new = max(m, rowmax), P = 2^(S2 - m_new), r = 2^(m - m_new);
//   P^ = HIF4(P) in registers: the lane's 32 keys are 8 complete 4-key blocks,
//     8-key blocks pair with lane l^32; values become FP6 operands directly;
//   O^T[d, q] += V^T P^T: the lane's P^ values already form the B operand of
//     the 32x32x64 MFMA (the pre-pass stored V^ in the matching key order), an
//     fp32 epilogue applies b_P*b_V; the normalizer comes out of one more
//     MFMA against an all-ones A operand (the [V^ | 1] column of the paper).
#include "hifa4_device.h"
#include "hifa4_internal.h"

namespace hifa4 {

struct TileMap {
  int b, hq, hk, qw, L, t0, nJ;
  bool active;       // this wave has query rows inside the sequence
  bool wg_live;      // the workgroup has work
};

__device__ __forceinline__ TileMap map_tile(const AttnArgs& a, int heads_per_wg, int qsub, int n_qtiles) {
  TileMap m;
  const int n_hgroups = a.hq / heads_per_wg;
  const int per_qt = n_hgroups * a.batch;
  const int item = blockIdx.x;
  const int qt = n_qtiles - 1 - item / per_qt;        // longest first
  const int rem = item % per_qt;
  const int hg = rem % n_hgroups;
  m.b = rem / n_hgroups;
  const int wave = threadIdx.x >> 6;
  m.hq = hg * heads_per_wg + wave / qsub;
  m.hk = m.hq / (a.hq / a.hkv);
  const int span = 32 * qsub;
  m.t0 = a.cu ? a.cu[m.b] : m.b * a.S;
  m.L = a.cu ? a.cu[m.b + 1] - m.t0 : a.S;
  const int q0 = qt * span;
  m.wg_live = q0 < m.L;
  m.qw = q0 + 32 * (wave % qsub);
  m.active = m.qw < m.L;
  const int qend = min(q0 + span, m.L);
  m.nJ = m.wg_live ? (qend - 1) / 64 + 1 : 0;
  return m;
}

typedef uint32_t u4_t __attribute__((ext_vector_type(4)));
typedef float f4_t __attribute__((ext_vector_type(4)));

// Copy one pre-pass chunk (bytes multiple of 16) from global memory to LDS.
__device__ __forceinline__ void stage_chunk(uint8_t* lds, const uint8_t* __restrict__ g, int bytes) {
  const u4_t* src = reinterpret_cast<const u4_t*>(g);
  u4_t* dst = reinterpret_cast<u4_t*>(lds);
  for (int i = threadIdx.x; i < bytes / 16; i += blockDim.x) dst[i] = src[i];
}

__device__ __forceinline__ i8_t ld_op6(const uint8_t* p) {
  const uint2* q = reinterpret_cast<const uint2*>(p);
  const uint2 a = q[0], b = q[1], c = q[2];
  i8_t r;
  r[0] = (int)a.x; r[1] = (int)a.y; r[2] = (int)b.x; r[3] = (int)b.y; r[4] = (int)c.x; r[5] = (int)c.y;
  r[6] = 0; r[7] = 0;
  return r;
}

__device__ __forceinline__ f16v_t mfma6(const i8_t& A, const i8_t& B, const f16v_t& C) {
  // FP6 E2M3 x FP6 E2M3, unit E8M0 scales (127 = 2^0).
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(A, B, C, 2, 2, 0, 127, 0, 127);
}

__device__ __forceinline__ half_t hmax(half_t a, half_t b) { return a > b ? a : b; }

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
  return __builtin_elementwise_max(__builtin_bit_cast(h2_t, p.x), __builtin_bit_cast(h2_t, p.y));
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

// t = fp16(p*R + C) for both halves of p (fp16), R and C fp32: each result is
// the exact fused value rounded once to fp16.
__device__ __forceinline__ h2_t fma_grid2(h2_t p, float R, float C) {
  h2_t y;
  asm("v_fma_mixlo_f16 %0, %1, %2, %3 op_sel_hi:[1,0,0]\n\t"
      "v_fma_mixhi_f16 %0, %1, %2, %3 op_sel:[1,0,0] op_sel_hi:[1,0,0]"
      : "=&v"(y)
      : "v"(p), "v"(R), "v"(C));
  return y;
}

// Global key index (within the 64-key block) held by lane half h at tile t,
// accumulator register v of the 32x32 output layout.
__device__ __forceinline__ int key_of(int t, int h, int v) { return 32 * t + 8 * (v >> 2) + 4 * h + (v & 3); }

// ---------------------------------------------------------------------------
// HiFA4 kernel.
//
// Pipeline per wave: the QK^T MFMAs of block J+1 are issued before the
// softmax / quantization VALU work of block J, so the matrix cores and the
// vector ALUs overlap.  K/V chunks rotate through three LDS buffers: while
// block J is consumed (K of J+1, V of J), chunk J+2 is fetched into registers
// and written to the buffer chunk J-1 used.
//
// Deferred rescale: instead of O <- r*O every block, the kernel keeps
// O* = O / rho and l* = l / rho with rho the product of the rescale factors so
// far, and adds each block's contribution scaled by 1/rho.  O*/l* = O/l, so
// the output and the P^ codes are unchanged; only the fp32 rounding of O
// differs.  A factor r = 0 (a running max that grows by more than 24 in log2
// units after the first block) wipes the history, exactly as r*O does.
template <int G, int NORM, bool DEBUG>
__global__ void __launch_bounds__(256, (G == 1 ? 2 : 1)) k_attn_hif4(AttnArgs a, int heads_per_wg, int qsub, int n_qtiles) {
  constexpr int D = 64 * G;
  constexpr int DT = D / 32;
  constexpr ChunkLayout lay = chunk_layout_hif4(G);
  constexpr int cbytes = (int)lay.bytes;
  constexpr int n16 = cbytes / 16;
  constexpr int n_pre = (n16 + 255) / 256;
  constexpr bool kPipe = G <= 2;
  extern __shared__ __align__(16) uint8_t smem[];
  const TileMap tm = map_tile(a, heads_per_wg, qsub, n_qtiles);
  if (!tm.wg_live) return;
  const int lane = threadIdx.x & 63, h = lane >> 5, col = lane & 31;
  const int qi = tm.qw + col;
  const bool row_ok = tm.active && qi < tm.L;
  const int jw_last = tm.active ? (min(tm.qw + 31, tm.L - 1)) / 64 : -1;

  // ---- Q tile: Smooth-QK (fp16(q*s)) then HIF4 into FP6 B operands.
  i8_t qop[G];
  float bq[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    float x[32];
    if (row_ok) {
      const half_t* src = a.q + ((size_t)(tm.t0 + qi) * a.hq + tm.hq) * D + 64 * g + 32 * h;
      const u4_t* p = reinterpret_cast<const u4_t*>(src);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const u4_t w = p[v];
        const h8_t hh = __builtin_bit_cast(h8_t, w);
#pragma unroll
        for (int i = 0; i < 8; ++i) x[8 * v + i] = (float)hh[i];
      }
      if (a.s) {
        const float* sp = a.s + (size_t)tm.hk * D + 64 * g + 32 * h;
#pragma unroll
        for (int c = 0; c < 32; ++c) x[c] = (float)mul_rn16(x[c], sp[c]);
      }
    } else {
#pragma unroll
      for (int c = 0; c < 32; ++c) x[c] = 0.0f;
    }
    float a4own[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      float mm = fabsf(x[4 * k]);
#pragma unroll
      for (int i = 1; i < 4; ++i) mm = fmaxf(mm, fabsf(x[4 * k + i]));
      a4own[k] = mm;
    }
    float a4_all[16];
    gather_a4<kRows>(a4own, a4_all, h);
    const GroupMeta gm = group_meta(a4_all);
    const float R = hif4_rcp_step(gm.base);
    h32_t hv;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float C = round_const(block_shift(gm, 8 * h + k));
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float xv = x[4 * k + i];
        const float ov = hif4_elem(fabsf(xv), R, C);
        hv[4 * k + i] = (half_t)(xv < 0.0f ? -ov : ov);
      }
    }
    const i6_t pk = __builtin_amdgcn_cvt_scalef32_pk32_fp6_f16(hv, 1.0f);
#pragma unroll
    for (int i = 0; i < 6; ++i) qop[g][i] = pk[i];
    qop[g][6] = 0;
    qop[g][7] = 0;
    bq[g] = 0.25f * gm.b;
  }

  i8_t ones;
  {
    uint32_t w[6] = {0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int s = 0; s < 32; ++s) {
      const int bit = 6 * s;
      w[bit >> 5] |= kE2M3One << (bit & 31);
      if ((bit & 31) > 26) w[(bit >> 5) + 1] |= kE2M3One >> (32 - (bit & 31));
    }
#pragma unroll
    for (int i = 0; i < 6; ++i) ones[i] = (int)w[i];
    ones[6] = 0;
    ones[7] = 0;
  }

  f16v_t O[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) O[dt][v] = 0.0f;
  half_t m_run = (half_t)(-__builtin_inff());
  float l_star = 0.0f;     // l / rho (consistent or mismatched per NORM)
  float inv_rho = 1.0f;    // 1 / rho

  const uint8_t* ws_base = a.ws + ((size_t)(tm.b * a.hkv + tm.hk) * a.NB) * lay.bytes;
  stage_chunk(smem, ws_base, cbytes);
  if (tm.nJ > 1) stage_chunk(smem + cbytes, ws_base + cbytes, cbytes);
  __syncthreads();

  // QK MFMAs of one block: acc[t][g] = K^ tile (t, g) x Q^ group g.
  f16v_t acc[2][G];
  auto issue_qk = [&](const uint8_t* buf) {
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const i8_t kop = ld_op6(buf + lay.k_op + ((size_t)(t * G + g) * 64 + lane) * 24);
        const f16v_t zero = {};
        acc[t][g] = mfma6(kop, qop[g], zero);
      }
  };
  if (kPipe && tm.active) issue_qk(smem);

  for (int J = 0; J < tm.nJ; ++J) {
    const uint8_t* cur = smem + (J % 3) * cbytes;
    const bool has_next2 = J + 2 < tm.nJ;
    u4_t pre[n_pre];
    {
      const u4_t* src = reinterpret_cast<const u4_t*>(ws_base + (size_t)(has_next2 ? J + 2 : J) * cbytes);
#pragma unroll
      for (int r = 0; r < n_pre; ++r) {
        const int i = threadIdx.x + 256 * r;
        pre[r] = src[i < n16 ? i : n16 - 1];
      }
    }
    if (tm.active && J <= jw_last) {
      if (!kPipe) issue_qk(cur);
      // ---- scores: S2 = fp16((sum_g t_g) * c), t_g = acc_g * (b_q b_k) exact.
      h2_t s2[2][8];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        float sacc[16];
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const float* ksc = reinterpret_cast<const float*>(cur + lay.k_scale) + (t * G + g) * 32 + 4 * h;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const f4_t bkv = *reinterpret_cast<const f4_t*>(ksc + 8 * j);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int v = 4 * j + i;
              const float w = bq[g] * bkv[i];
              sacc[v] = (g == 0) ? acc[t][g][v] * w : __builtin_fmaf(acc[t][g][v], w, sacc[v]);
            }
          }
        }
#pragma unroll
        for (int v2 = 0; v2 < 8; ++v2) s2[t][v2] = mul2_rn16(sacc[2 * v2], sacc[2 * v2 + 1], a.c);
      }
      // ---- issue the next block's QK^T while this block's VALU work runs.
      if (kPipe && J < jw_last) issue_qk(smem + ((J + 1) % 3) * cbytes);
      // ---- causal mask on the block that holds the diagonal.
      if (J == jw_last) {
        const half_t ninf = (half_t)(-__builtin_inff());
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int v = 0; v < 16; ++v)
            if (64 * J + key_of(t, h, v) > qi) s2[t][v >> 1][v & 1] = ninf;
      }
      // ---- running max (FP16), exchanged with lane l^32.
      h2_t mx2 = s2[0][0];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int v2 = 0; v2 < 8; ++v2) mx2 = __builtin_elementwise_max(mx2, s2[t][v2]);
      mx2 = max_with_partner(mx2);
      const half_t mx = hmax(mx2[0], mx2[1]);
      const half_t m_new = hmax(m_run, mx);
      const h2_t mn2 = {m_new, m_new};
      // ---- P = 2^(S2 - m_new), r = 2^(m - m_new), block max A = 2^(mx - m_new).
      h2_t p2[2][8];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int v2 = 0; v2 < 8; ++v2) p2[t][v2] = exp2_h2(s2[t][v2] - mn2);
      const h2_t ra = exp2_h2(h2_t{(half_t)(m_run - m_new), (half_t)(mx - m_new)});
      const float r = (float)ra[0];
      const float A = (float)ra[1];
      m_run = m_new;

      float psum = 0.0f;
      if (NORM == 1) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int v2 = 0; v2 < 8; ++v2) psum = __builtin_amdgcn_fdot2(p2[t][v2], h2_t{(half_t)1, (half_t)1}, psum, false);
        psum = add_with_partner(psum);
      }

      // ---- P^ = HIF4(P) over the block's 64 keys (P-Reordering).
      // Lane 4-block (t, j): keys 32t + 8j + 4h + [0,4) = p2[t][2j], p2[t][2j+1].
      h2_t a4p[4];          // own 4-block maxima, packed (t,0|t,1), (t,2|t,3)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int jp = 0; jp < 2; ++jp) {
          const h2_t m0 = __builtin_elementwise_max(p2[t][4 * jp], p2[t][4 * jp + 1]);
          const h2_t m1 = __builtin_elementwise_max(p2[t][4 * jp + 2], p2[t][4 * jp + 3]);
          a4p[2 * t + jp] = h2_t{hmax(m0[0], m0[1]), hmax(m1[0], m1[1])};
        }
      const uint32_t base = e6m2_ceil(A);
      const float bval = e6m2_value(base);
      const float R = hif4_rcp_step(base);
      // fp16 floors of the half and quarter ranges: an fp16 value x satisfies
      // x <= 0.875b iff x <= floor16(0.875b) (round-toward-zero conversion).
      const h2_t thr = __builtin_bit_cast(h2_t, __builtin_amdgcn_cvt_pkrtz(0.875f * bval, 0.4375f * bval));
      uint32_t e2bits = 0, e3bits = 0;
      h2_t cpair[8];        // per 4-block rounding constant (fp16, both halves)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const h2_t a8 = max_with_partner(a4p[q]);
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const int t = q >> 1, j = 2 * (q & 1) + e;
          const bool e2 = a8[e] <= thr[0];
          const bool e3 = a4p[q][e] <= (e2 ? thr[1] : thr[0]);
          const int sh = (int)e2 + (int)e3;
          // C16 = 1.5 * 2^(10-sh) as fp16: exponent field 25 - sh, mantissa 0x200
          const uint16_t cb = (uint16_t)(((25 - sh) << 10) | 0x200);
          const half_t c16 = __builtin_bit_cast(half_t, cb);
          cpair[4 * t + j] = h2_t{c16, c16};
          if (DEBUG) {
            e2bits |= (uint32_t)e2 << (4 * t + j);
            e3bits |= (uint32_t)e3 << (8 * t + 2 * j + h);
            const bool e3o = partner_h2(a4p[q], h)[e] <= (e2 ? thr[1] : thr[0]);
            e3bits |= (uint32_t)e3o << (8 * t + 2 * j + (h ^ 1));
          }
        }
      }
      // o = u * 2^-sh: round P*R onto the grid 2^-sh in one fp16 fma, then
      // subtract the offset (both exact); then pack 32 values to FP6.
      h32_t ov;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const h2_t c2 = cpair[4 * t + j];
#pragma unroll
          for (int e = 0; e < 2; ++e) {
            const h2_t pv = p2[t][2 * j + e];
            h2_t tt = fma_grid2(pv, R, (float)c2[0]);
            tt = tt - c2;
            // slot order of the B operand: slot 2v + t holds tile t, reg v
            const int v0 = 4 * j + 2 * e;
            ov[2 * v0 + t] = tt[0];
            ov[2 * (v0 + 1) + t] = tt[1];
          }
        }
      const i6_t pk = __builtin_amdgcn_cvt_scalef32_pk32_fp6_f16(ov, 1.0f);
      i8_t pop;
#pragma unroll
      for (int i = 0; i < 6; ++i) pop[i] = pk[i];
      pop[6] = 0;
      pop[7] = 0;

      if (DEBUG && row_ok) {
        uint8_t* dc = a.dbg_codes + (((size_t)tm.hq * a.total_tokens + tm.t0 + qi) * a.NB + J) * 32;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int q4 = 8 * t + 2 * j + h;
            const int sh = (int)((e2bits >> (4 * t + j)) & 1u) + (int)((e3bits >> q4) & 1u);
            uint32_t nib[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int v = 4 * j + i;
              nib[i] = (uint32_t)((float)ov[2 * v + t] * (float)(1 << sh));
            }
            dc[16 * t + 4 * j + 2 * h] = (uint8_t)(nib[0] | (nib[1] << 4));
            dc[16 * t + 4 * j + 2 * h + 1] = (uint8_t)(nib[2] | (nib[3] << 4));
          }
        if (h == 0)
          a.dbg_meta[((size_t)tm.hq * a.total_tokens + tm.t0 + qi) * a.NB + J] = base | (e2bits << 8) | (e3bits << 16);
      }

      // ---- deferred rescale bookkeeping (lane-uniform factors).
      if (J > 0 && __builtin_amdgcn_ballot_w64(r == 0.0f) != 0) {
        // history wiped for some rows: O <- 0*O, l <- 0*l there
        if (r == 0.0f) {
#pragma unroll
          for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int v = 0; v < 16; ++v) O[dt][v] = 0.0f;
          l_star = 0.0f;
        }
      }
      inv_rho = (r == 0.0f) ? 1.0f : inv_rho * __builtin_amdgcn_rcpf(r);
      if (__builtin_amdgcn_ballot_w64(inv_rho > 0x1p64f) != 0) {
        const float rho = __builtin_amdgcn_rcpf(inv_rho);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int v = 0; v < 16; ++v) O[dt][v] *= rho;
        l_star *= rho;
        inv_rho = 1.0f;
      }
      const float wp = 0.25f * bval * inv_rho;      // b_P/4 / rho
      // ---- [O | l] += P^ [V^ | 1]; V^'s scale is split over three MFMAs.
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const i8_t vop = ld_op6(cur + lay.v_op + ((size_t)dt * 64 + lane) * 24);
        const int vs = reinterpret_cast<const int*>(cur + lay.v_scale)[32 * dt + col];
        f16v_t pv = {};
        pv = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(vop, pop, pv, 2, 2, 0, vs, 0, 127);
        pv = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(vop, pop, pv, 2, 2, 1, vs, 0, 127);
        pv = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(vop, pop, pv, 2, 2, 2, vs, 0, 127);
#pragma unroll
        for (int v = 0; v < 16; ++v) O[dt][v] = __builtin_fmaf(pv[v], wp, O[dt][v]);
      }
      if (NORM == 1) {
        l_star = __builtin_fmaf(psum, inv_rho, l_star);
      } else {
        const f16v_t zero = {};
        const f16v_t lacc = mfma6(ones, pop, zero);
        l_star = __builtin_fmaf(lacc[0], wp, l_star);
      }
    }
    if (has_next2) {
      u4_t* dst = reinterpret_cast<u4_t*>(smem + ((J + 2) % 3) * cbytes);
#pragma unroll
      for (int r = 0; r < n_pre; ++r) {
        const int i = threadIdx.x + 256 * r;
        if (i < n16) dst[i] = pre[r];
      }
    }
    __syncthreads();
  }

  // ---- finalize: O = fp16(O*/l*), LSE = m ln2 + ln(l* rho).
  if (row_ok) {
    const float inv = 1.0f / l_star;
    half_t* dst = a.o + ((size_t)(tm.t0 + qi) * a.hq + tm.hq) * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        typedef _Float16 h4_t __attribute__((ext_vector_type(4)));
        h4_t o4;
#pragma unroll
        for (int i = 0; i < 4; ++i) o4[i] = (half_t)(O[dt][4 * j + i] * inv);
        *reinterpret_cast<h4_t*>(dst + 32 * dt + 8 * j + 4 * h) = o4;
      }
    if (h == 0)
      a.lse[(size_t)tm.hq * a.total_tokens + tm.t0 + qi] =
          (float)m_run * 0.69314718055994531f + logf(l_star) - logf(inv_rho);
  }
}

// ---------------------------------------------------------------------------
// FP16-operand variant (the C16V16 reference): same decomposition and softmax,
// 32x32x16 f16 MFMAs, P in fp16 as the PV operand, O accumulated by the MFMA,
// l = rowsum(P).
template <int D>
__global__ void __launch_bounds__(256) k_attn_fp16(AttnArgs a, int heads_per_wg, int qsub, int n_qtiles) {
  constexpr int KC = D / 16;
  constexpr int DT = D / 32;
  constexpr ChunkLayout lay = chunk_layout_fp16(D);
  extern __shared__ __align__(16) uint8_t smem[];
  const TileMap tm = map_tile(a, heads_per_wg, qsub, n_qtiles);
  if (!tm.wg_live) return;
  const int lane = threadIdx.x & 63, h = lane >> 5, col = lane & 31;
  const int qi = tm.qw + col;
  const bool row_ok = tm.active && qi < tm.L;
  const int jw_last = tm.active ? (min(tm.qw + 31, tm.L - 1)) / 64 : -1;

  h8_t qf[KC];
#pragma unroll
  for (int kc = 0; kc < KC; ++kc) {
    if (row_ok)
      qf[kc] = *reinterpret_cast<const h8_t*>(a.q + ((size_t)(tm.t0 + qi) * a.hq + tm.hq) * D + 16 * kc + 8 * h);
    else
      for (int e = 0; e < 8; ++e) qf[kc][e] = (half_t)0.0f;
  }
  f16v_t O[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) O[dt][v] = 0.0f;
  half_t m_run = (half_t)(-__builtin_inff());
  float l_sum = 0.0f;

  const uint8_t* ws_base = a.ws + ((size_t)(tm.b * a.hkv + tm.hk) * a.NB) * lay.bytes;
  constexpr int cbytes = (int)lay.bytes;
  stage_chunk(smem, ws_base, cbytes);
  __syncthreads();

  for (int J = 0; J < tm.nJ; ++J) {
    const uint8_t* cur = smem + (J & 1) * cbytes;
    const bool has_next = J + 1 < tm.nJ;
    if (tm.active && J <= jw_last) {
      h2_t s2[2][8];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        f16v_t acc = {};
#pragma unroll
        for (int kc = 0; kc < KC; ++kc) {
          const h8_t kf = *reinterpret_cast<const h8_t*>(cur + lay.k_op + ((size_t)(t * KC + kc) * 64 + lane) * 16);
          acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(kf, qf[kc], acc, 0, 0, 0);
        }
#pragma unroll
        for (int v2 = 0; v2 < 8; ++v2) {
          s2[t][v2][0] = (half_t)(acc[2 * v2] * a.c);
          s2[t][v2][1] = (half_t)(acc[2 * v2 + 1] * a.c);
        }
      }
      if (64 * J + 63 > tm.qw) {
        const half_t ninf = (half_t)(-__builtin_inff());
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int v = 0; v < 16; ++v)
            if (64 * J + key_of(t, h, v) > qi) s2[t][v >> 1][v & 1] = ninf;
      }
      h2_t mx2 = s2[0][0];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int v2 = 0; v2 < 8; ++v2) mx2 = __builtin_elementwise_max(mx2, s2[t][v2]);
      half_t mx = hmax(mx2[0], mx2[1]);
      mx = hmax(mx, (half_t)shfl_xor32((float)mx));
      const half_t m_new = hmax(m_run, mx);
      const h2_t mn2 = {m_new, m_new};
      h2_t p2[2][8];
      float ps = 0.0f;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int v2 = 0; v2 < 8; ++v2) {
          p2[t][v2] = exp2_h2(s2[t][v2] - mn2);
          ps += (float)p2[t][v2][0] + (float)p2[t][v2][1];
        }
      ps += shfl_xor32(ps);
      const h2_t rr = exp2_h2(h2_t{(half_t)(m_run - m_new), (half_t)0});
      const float r = (float)rr[0];
      m_run = m_new;
      l_sum = l_sum * r + ps;
      if (__builtin_amdgcn_ballot_w64(r != 1.0f) != 0) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int v = 0; v < 16; ++v) O[dt][v] *= r;
      }
      // B operand chunks: c = 2t + jp holds p2[t][4jp .. 4jp+3] (keys
      // 32t + 8(2jp + e/4) + 4h + e%4 at slot e).
      h8_t pb[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int t = c >> 1, jp = c & 1;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          pb[c][2 * e] = p2[t][4 * jp + e][0];
          pb[c][2 * e + 1] = p2[t][4 * jp + e][1];
        }
      }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const h8_t vf = *reinterpret_cast<const h8_t*>(cur + lay.v_op + ((size_t)(dt * 4 + c) * 64 + lane) * 16);
          O[dt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vf, pb[c], O[dt], 0, 0, 0);
        }
    }
    if (has_next) stage_chunk(smem + ((J + 1) & 1) * cbytes, ws_base + (size_t)(J + 1) * cbytes, cbytes);
    __syncthreads();
  }
  if (row_ok) {
    const float inv = 1.0f / l_sum;
    half_t* dst = a.o + ((size_t)(tm.t0 + qi) * a.hq + tm.hq) * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        typedef _Float16 h4_t __attribute__((ext_vector_type(4)));
        h4_t ov;
#pragma unroll
        for (int i = 0; i < 4; ++i) ov[i] = (half_t)(O[dt][4 * j + i] * inv);
        *reinterpret_cast<h4_t*>(dst + 32 * dt + 8 * j + 4 * h) = ov;
      }
    if (h == 0) a.lse[(size_t)tm.hq * a.total_tokens + tm.t0 + qi] = (float)m_run * 0.69314718055994531f + logf(l_sum);
  }
}

// ---------------------------------------------------------------------------
template <typename K>
static hipError_t launch_k(K kern, const AttnArgs& a, size_t lds, hipStream_t st) {
  const int grp = a.hq / a.hkv;
  const int heads_per_wg = (grp % 4 == 0) ? 4 : ((grp % 2 == 0) ? 2 : 1);
  const int qsub = 4 / heads_per_wg;
  const int span = 32 * qsub;
  const int n_qtiles = (a.S + span - 1) / span;
  const long n_items = (long)n_qtiles * (a.hq / heads_per_wg) * a.batch;
  if (n_items == 0) return hipSuccess;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds);
  if (e != hipSuccess) return e;
  kern<<<dim3((unsigned)n_items), dim3(256), lds, st>>>(a, heads_per_wg, qsub, n_qtiles);
  return hipGetLastError();
}

hipError_t launch_attention(const AttnArgs& a, int norm, bool fp16, hipStream_t st) {
  if (fp16) {
    const size_t lds = 2 * chunk_layout_fp16(a.D).bytes;
    switch (a.D) {
      case 64: return launch_k(k_attn_fp16<64>, a, lds, st);
      case 128: return launch_k(k_attn_fp16<128>, a, lds, st);
      case 256: return launch_k(k_attn_fp16<256>, a, lds, st);
    }
    return hipErrorInvalidValue;
  }
  const size_t lds = 3 * chunk_layout_hif4(a.D / 64).bytes;
  const bool dbg = a.dbg_codes != nullptr;
#define HIFA4_DISPATCH(G)                                                                            \
  do {                                                                                               \
    if (norm == 0)                                                                                   \
      return dbg ? launch_k(k_attn_hif4<G, 0, true>, a, lds, st) : launch_k(k_attn_hif4<G, 0, false>, a, lds, st); \
    return dbg ? launch_k(k_attn_hif4<G, 1, true>, a, lds, st) : launch_k(k_attn_hif4<G, 1, false>, a, lds, st);   \
  } while (0)
  switch (a.D) {
    case 64: HIFA4_DISPATCH(1);
    case 128: HIFA4_DISPATCH(2);
    case 256: HIFA4_DISPATCH(4);
  }
#undef HIFA4_DISPATCH
  return hipErrorInvalidValue;
}

}  // namespace hifa4
