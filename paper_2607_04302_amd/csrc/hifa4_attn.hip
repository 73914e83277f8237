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

// Global key index (within the 64-key block) held by lane half h at tile t,
// accumulator register v of the 32x32 output layout.
__device__ __forceinline__ int key_of(int t, int h, int v) { return 32 * t + 8 * (v >> 2) + 4 * h + (v & 3); }

// ---------------------------------------------------------------------------
template <int G, int NORM>
__global__ void __launch_bounds__(256) k_attn_hif4(AttnArgs a, int heads_per_wg, int qsub, int n_qtiles) {
  constexpr int D = 64 * G;
  constexpr int DT = D / 32;
  constexpr ChunkLayout lay = chunk_layout_hif4(G);
  constexpr int cbytes = (int)lay.bytes;
  constexpr int n16 = cbytes / 16;
  constexpr int n_pre = n16 < 1024 ? (n16 + 255) / 256 : 4;
  extern __shared__ __align__(16) uint8_t smem[];
  const TileMap tm = map_tile(a, heads_per_wg, qsub, n_qtiles);
  if (!tm.wg_live) return;
  const int lane = threadIdx.x & 63, h = lane >> 5, col = lane & 31;
  const int qi = tm.qw + col;                 // this lane's query position
  const bool row_ok = tm.active && qi < tm.L;
  const int jw_last = tm.active ? (min(tm.qw + 31, tm.L - 1)) / 64 : -1;

  // ---- Q tile: Smooth-QK then HIF4 into FP6 B operands (one per group).
  i8_t qop[G];
  float bq[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    float x[32], o[32];
    if (row_ok) {
      const half_t* src = a.q + ((size_t)(tm.t0 + qi) * a.hq + tm.hq) * D + 64 * g + 32 * h;
      const uint4* p = reinterpret_cast<const uint4*>(src);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        uint4 w = p[v];
        const half_t* hh = reinterpret_cast<const half_t*>(&w);
#pragma unroll
        for (int i = 0; i < 8; ++i) x[8 * v + i] = (float)hh[i];
      }
      if (a.s) {
        const float* sp = a.s + (size_t)tm.hk * D + 64 * g + 32 * h;
#pragma unroll
        for (int c = 0; c < 32; ++c) x[c] = (float)(half_t)(x[c] * sp[c]);
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
        o[4 * k + i] = xv < 0.0f ? -ov : ov;
        hv[4 * k + i] = (half_t)o[4 * k + i];
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
    // 32 FP6 fields of 1.0 packed in 192 bits.
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
  float l_con = 0.0f, l_mis = 0.0f;

  const uint8_t* ws_base = a.ws + ((size_t)(tm.b * a.hkv + tm.hk) * a.NB) * lay.bytes;
  stage_chunk(smem, ws_base, cbytes);
  __syncthreads();

  for (int J = 0; J < tm.nJ; ++J) {
    // Prefetch (up to 16 KB of) the next chunk into registers while this one
    // is consumed; the index is clamped so every load stays inside the chunk.
    // The loads are unconditional (the last iteration re-reads its own chunk)
    // so that the staging registers never live in scratch memory.
    const bool has_next = J + 1 < tm.nJ;
    u4_t pre[n_pre];
    {
      const u4_t* src = reinterpret_cast<const u4_t*>(ws_base + (size_t)(has_next ? J + 1 : J) * cbytes);
#pragma unroll
      for (int r = 0; r < n_pre; ++r) {
        const int i = threadIdx.x + 256 * r;
        pre[r] = src[i < n16 ? i : n16 - 1];
      }
    }
    const uint8_t* cur = smem + (J & 1) * cbytes;
    if (tm.active && J <= jw_last) {
      // ---- S^T = K^ Q^T (exact group dots) and the fp32 score epilogue.
      h2_t s2[2][8];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        f16v_t sacc;
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const i8_t kop = ld_op6(cur + lay.k_op + ((size_t)(t * G + g) * 64 + lane) * 24);
          f16v_t zero = {};
          const f16v_t acc = mfma6(kop, qop[g], zero);
          const float* ksc = reinterpret_cast<const float*>(cur + lay.k_scale) + (t * G + g) * 32 + 4 * h;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const f4_t bkv = *reinterpret_cast<const f4_t*>(ksc + 8 * j);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int v = 4 * j + i;
              const float w = bq[g] * bkv[i];
              sacc[v] = (g == 0) ? acc[v] * w : __builtin_fmaf(acc[v], w, sacc[v]);
            }
          }
        }
#pragma unroll
        for (int v2 = 0; v2 < 8; ++v2) {
          s2[t][v2][0] = (half_t)(sacc[2 * v2] * a.c);
          s2[t][v2][1] = (half_t)(sacc[2 * v2 + 1] * a.c);
        }
      }
      // ---- causal mask (only the block that holds the diagonal).
      if (64 * J + 63 > tm.qw) {
        const half_t ninf = (half_t)(-__builtin_inff());
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int v = 0; v < 16; ++v)
            if (64 * J + key_of(t, h, v) > qi) s2[t][v >> 1][v & 1] = ninf;
      }
      // ---- running max (FP16).
      h2_t mx2 = s2[0][0];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int v2 = 0; v2 < 8; ++v2) mx2 = __builtin_elementwise_max(mx2, s2[t][v2]);
      half_t mx = hmax(mx2[0], mx2[1]);
      {
        const float other = shfl_xor32((float)mx);
        mx = hmax(mx, (half_t)other);
      }
      const half_t m_new = hmax(m_run, mx);
      const h2_t mn2 = {m_new, m_new};
      // ---- P = 2^(S2 - m_new) in fp16; r = 2^(m - m_new).
      h2_t p2[2][8];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int v2 = 0; v2 < 8; ++v2) p2[t][v2] = exp2_h2(s2[t][v2] - mn2);
      const h2_t rr = exp2_h2(h2_t{(half_t)(m_run - m_new), (half_t)0});
      const float r = (float)rr[0];
      m_run = m_new;

      if (NORM == 1) {
        float ps = 0.0f;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int v2 = 0; v2 < 8; ++v2) ps += (float)p2[t][v2][0] + (float)p2[t][v2][1];
        ps += shfl_xor32(ps);
        l_mis = l_mis * r + ps;
      }

      // ---- P^ = HIF4(P) over the block's 64 keys (P-Reordering).
      // The lane's 4-block (t, j) holds keys 32t + 8j + 4h + [0,4): global
      // 4-block index 8t + 2j + h; its values are p2[t][2j], p2[t][2j+1].
      float a4own[8];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const h2_t mm = __builtin_elementwise_max(p2[t][2 * j], p2[t][2 * j + 1]);
          a4own[4 * t + j] = (float)hmax(mm[0], mm[1]);
        }
      float a4_all[16];
      gather_a4<kKeys>(a4own, a4_all, h);
      const GroupMeta gm = group_meta(a4_all);
      const float R = hif4_rcp_step(gm.base);
      f16v_t px, py;     // tile 0 -> x, tile 1 -> y (the cvt interleaves them)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float C = round_const(block_shift(gm, 8 * t + 2 * j + h));
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int v = 4 * j + i;
            const float pv = (float)p2[t][v >> 1][v & 1];
            const float ov = hif4_elem(pv, R, C);
            if (t == 0) px[v] = ov; else py[v] = ov;
          }
        }
      const i6_t pk = __builtin_amdgcn_cvt_scalef32_2xpk16_fp6_f32(px, py, 1.0f);
      i8_t pop;
#pragma unroll
      for (int i = 0; i < 6; ++i) pop[i] = pk[i];
      pop[6] = 0;
      pop[7] = 0;
      const float bp = 0.25f * gm.b;

      if (a.dbg_codes && row_ok) {
        // canonical dump: byte index = key/2; the lane writes the bytes of its
        // 4-blocks (keys 32t+8j+4h .. +3 -> bytes 16t+4j+2h, +1).
        uint8_t* dc = a.dbg_codes + (((size_t)tm.hq * a.total_tokens + tm.t0 + qi) * a.NB + J) * 32;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int sh = block_shift(gm, 8 * t + 2 * j + h);
            uint32_t nib[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float ov = t == 0 ? px[4 * j + i] : py[4 * j + i];
              nib[i] = (uint32_t)(ov * (float)(1 << sh));
            }
            dc[16 * t + 4 * j + 2 * h] = (uint8_t)(nib[0] | (nib[1] << 4));
            dc[16 * t + 4 * j + 2 * h + 1] = (uint8_t)(nib[2] | (nib[3] << 4));
          }
        if (h == 0)
          a.dbg_meta[((size_t)tm.hq * a.total_tokens + tm.t0 + qi) * a.NB + J] = gm.base | (gm.e2 << 8) | (gm.e3 << 16);
      }

      // ---- rescale history (skipped while the max is unchanged).
      const bool need = __builtin_amdgcn_ballot_w64(r != 1.0f) != 0;
      if (need) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int v = 0; v < 16; ++v) O[dt][v] *= r;
      }
      // ---- [O | l] += P^ [V^ | 1].
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const i8_t vop = ld_op6(cur + lay.v_op + ((size_t)dt * 64 + lane) * 24);
        f16v_t zero = {};
        const f16v_t acc = mfma6(vop, pop, zero);
        const float* vsc = reinterpret_cast<const float*>(cur + lay.v_scale) + 32 * dt + 4 * h;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const f4_t bvv = *reinterpret_cast<const f4_t*>(vsc + 8 * j);
#pragma unroll
          for (int i = 0; i < 4; ++i) O[dt][4 * j + i] = __builtin_fmaf(acc[4 * j + i], bp * bvv[i], O[dt][4 * j + i]);
        }
      }
      {
        f16v_t zero = {};
        const f16v_t lacc = mfma6(ones, pop, zero);
        l_con = l_con * r + bp * lacc[0];
      }
    }
    if (has_next) {
      u4_t* dst = reinterpret_cast<u4_t*>(smem + ((J + 1) & 1) * cbytes);
#pragma unroll
      for (int r = 0; r < n_pre; ++r) {
        const int i = threadIdx.x + 256 * r;
        if (i < n16) dst[i] = pre[r];
      }
      if (n16 > 1024) stage_chunk(smem + ((J + 1) & 1) * cbytes + 16384, ws_base + (size_t)(J + 1) * cbytes + 16384, cbytes - 16384);
    }
    __syncthreads();
  }

  // ---- finalize: O = fp16(O / l), LSE = m ln2 + ln l.
  if (row_ok) {
    const float l = NORM == 1 ? l_mis : l_con;
    const float inv = 1.0f / l;
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
    if (h == 0) a.lse[(size_t)tm.hq * a.total_tokens + tm.t0 + qi] = (float)m_run * 0.69314718055994531f + logf(l);
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
  const size_t lds = 2 * chunk_layout_hif4(a.D / 64).bytes;
  if (norm == 0) {
    switch (a.D) {
      case 64: return launch_k(k_attn_hif4<1, 0>, a, lds, st);
      case 128: return launch_k(k_attn_hif4<2, 0>, a, lds, st);
      case 256: return launch_k(k_attn_hif4<4, 0>, a, lds, st);
    }
  } else {
    switch (a.D) {
      case 64: return launch_k(k_attn_hif4<1, 1>, a, lds, st);
      case 128: return launch_k(k_attn_hif4<2, 1>, a, lds, st);
      case 256: return launch_k(k_attn_hif4<4, 1>, a, lds, st);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace hifa4
