// HIF4 quantization kernels: canonical Q^/K^/V^ outputs, the attention
// pre-pass that writes MFMA-ready K and V operands, calibration reductions,
// and the exponential self-test.
//
// Paper: Algorithm 1 (Smooth-QK step, HIF4 of Q, K, V); Eq. 1 (q*s, k/s
// after RoPE); Appendix C (GQA: s is per key-head channel).
#include "hifa4_device.h"
#include "hifa4_internal.h"
#include "hifa4_packed.h"

namespace hifa4 {

// Token index (row of the [T, H, D] view) of position i in sequence b.
__device__ __forceinline__ int seq_start(const int* cu, int b, int S) {
  return cu ? cu[b] : b * S;
}
// a length above max_seqlen is outside the contract; clamping it keeps every
// access inside the caller's buffers
__device__ __forceinline__ int seq_len(const int* cu, int b, int S) {
  return cu ? min(cu[b + 1] - cu[b], S) : S;
}

// Load 32 consecutive fp16 channels of one (token, head) row and apply the
// Smooth-QK scale: q~ = fp16(q*s) and k~ = fp16(k/s), the exact product or
// quotient rounded once.  Returns the values as fp32.
// For K, `rs` may hold the reciprocals RN32(1/s) of the same 32 channels;
// the quotient then comes from div_rn16_rcp (same result, mostly without a
// division).
template <bool kIsK>
__device__ __forceinline__ void load_smoothed32(const half_t* __restrict__ src,
                                                const float* __restrict__ s, float x[32],
                                                const float* rs = nullptr) {
  const uint4* p = reinterpret_cast<const uint4*>(src);
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    uint4 w = p[v];
    const half_t* h = reinterpret_cast<const half_t*>(&w);
#pragma unroll
    for (int i = 0; i < 8; ++i) x[8 * v + i] = (float)h[i];
  }
  if (s) {
    if (kIsK && rs) {
#pragma unroll
      for (int c = 0; c < 32; ++c) x[c] = (float)div_rn16_rcp(x[c], s[c], rs[c]);
    } else {
#pragma unroll
      for (int c = 0; c < 32; ++c) x[c] = (float)(kIsK ? div_rn16(x[c], s[c]) : mul_rn16(x[c], s[c]));
    }
  }
}

// Quantize 32 elements held as 8 complete 4-blocks (block order per LAYOUT);
// the partner lane (l^32) holds the other 16.  Outputs per element: o (the
// signed E2M3 value u*2^-sh) and the group metadata.
template <int LAYOUT>
__device__ __forceinline__ GroupMeta quantize_split(const float x[32], float o[32], int h) {
  float a4own[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    float m = fabsf(x[4 * k]);
#pragma unroll
    for (int i = 1; i < 4; ++i) m = fmaxf(m, fabsf(x[4 * k + i]));
    a4own[k] = m;
  }
  float a4_all[16];
  gather_a4<LAYOUT>(a4own, a4_all, h);
  const GroupMeta g = group_meta(a4_all);
  const float R = hif4_rcp_step(g.base);
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const float C = round_const(block_shift(g, own_block<LAYOUT>(k, h)));
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float a = fabsf(x[4 * k + i]);
      const float ov = hif4_elem(a, R, C);
      o[4 * k + i] = x[4 * k + i] < 0.0f ? -ov : ov;
    }
  }
  return g;
}

__device__ __forceinline__ uint32_t nibble_of(float o, int sh) {
  const float uf = fabsf(o) * (float)(1 << sh);
  const uint32_t u = (uint32_t)uf;
  return (u == 0u) ? 0u : (u | (o < 0.0f ? 8u : 0u));
}

// ---------------------------------------------------------------------------
// Canonical Q^ / K^ (hifa4_quantize_qk).  One lane pair per group: lane l
// holds channels [32h, 32h+32) of group g of row (token, head), h = l/32.
// Each wave covers 32 groups.
template <bool kIsK>
__global__ void __launch_bounds__(256) k_quant_rows(const half_t* __restrict__ x, const float* __restrict__ s,
                                                    uint8_t* __restrict__ codes, uint32_t* __restrict__ meta,
                                                    int n_groups, int heads, int heads_kv, int G) {
  const int lane = threadIdx.x & 63;
  const int h = lane >> 5;
  const int gidx = (blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6)) * 32 + (lane & 31);
  if (gidx >= n_groups) return;   // whole lane pairs exit together
  const int g = gidx % G;
  const int head = (gidx / G) % heads;
  const int D = 64 * G;
  const half_t* src = x + (size_t)gidx * 64 + 32 * h;
  const float* sp = s ? s + (size_t)(head / (heads / heads_kv)) * D + 64 * g + 32 * h : nullptr;
  float v[32], o[32];
  load_smoothed32<kIsK>(src, sp, v);
  const GroupMeta gm = quantize_split<kRows>(v, o, h);
  uint32_t words[4];
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    uint32_t acc = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int el = 8 * w + e;
      const int sh = block_shift(gm, 8 * h + el / 4);
      acc |= nibble_of(o[el], sh) << (4 * e);
    }
    words[w] = acc;
  }
  uint4* dst = reinterpret_cast<uint4*>(codes + (size_t)gidx * 32 + 16 * h);
  *dst = make_uint4(words[0], words[1], words[2], words[3]);
  if (h == 0) meta[gidx] = gm.base | (gm.e2 << 8) | (gm.e3 << 16);
}

// ---------------------------------------------------------------------------
// Canonical V^ (hifa4_quantize_v): group = 64 tokens of one (kv head,
// channel) column, aligned to the sequence start.  Lanes 0..31 of a wave take
// 32 consecutive channels for tokens [0,32) of the group, lanes 32..63 the
// same channels for tokens [32,64).
__global__ void __launch_bounds__(256) k_quant_v_canon(const half_t* __restrict__ v, const int* __restrict__ cu,
                                                       uint8_t* __restrict__ codes, uint32_t* __restrict__ meta,
                                                       int batch, int S, int NB, int heads_kv, int D) {
  const int lane = threadIdx.x & 63;
  const int h = lane >> 5;
  const long gidx = ((long)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6)) * 32 + (lane & 31);
  const long n_groups = (long)batch * NB * heads_kv * D;
  if (gidx >= n_groups) return;
  const int d = (int)(gidx % D);
  const int hk = (int)((gidx / D) % heads_kv);
  const int J = (int)((gidx / ((long)D * heads_kv)) % NB);
  const int b = (int)(gidx / ((long)D * heads_kv * NB));
  const int t0 = seq_start(cu, b, S);
  const int L = seq_len(cu, b, S);
  float x[32], o[32];
#pragma unroll
  for (int k = 0; k < 32; ++k) {
    const int pos = 64 * J + 32 * h + k;
    x[k] = pos < L ? (float)v[((size_t)(t0 + pos) * heads_kv + hk) * D + d] : 0.0f;
  }
  const GroupMeta gm = quantize_split<kRows>(x, o, h);
  uint32_t words[4];
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    uint32_t acc = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int el = 8 * w + e;
      acc |= nibble_of(o[el], block_shift(gm, 8 * h + el / 4)) << (4 * e);
    }
    words[w] = acc;
  }
  *reinterpret_cast<uint4*>(codes + (size_t)gidx * 32 + 16 * h) = make_uint4(words[0], words[1], words[2], words[3]);
  if (h == 0) meta[gidx] = gm.base | (gm.e2 << 8) | (gm.e3 << 16);
}

// ---------------------------------------------------------------------------
// Attention pre-pass (HIF4 operands).  Two workgroups of 2G waves per
// (sequence b, kv head, 64-key block J): in the K workgroup wave w quantizes
// K half-tile t = w/G, group g = w%G; in the V workgroup wave w quantizes V
// channel tile w.
// Writes, for the chunk:
//   K operands [2 halves][G groups][2] operand records (64 lanes x dwords
//     0..3, then 64 lanes x dwords 4..5 of the lane's 6): lane l holds key
//     32t + l%32 and channels 64g + 32(l/32) + [0,32) in FP6 E2M3, i.e. the
//     A operand of S^T = K^ Q^T for the 32x32x64 MFMA, as the two operands of
//     the key's split base (below);
//   K scale words [2][G][32]: their two E8M0 bytes per key and group;
//   V operands [D/32 tiles][2] operand records: lane l holds channel
//     32dt + l%32 and, at FP6 slot s, the key 32(s/16) + 8((s%16)/4) +
//     4(l/32) + s%4 -- the key order in which the attention kernel's P^
//     operand arrives (the S^T accumulator registers of both 32-key halves in
//     order) -- again as the two operands of the split base;
//   V scale words [D]: their two E8M0 bytes per channel.
// Two-operand form of a HIF4 group for the FP6 MFMA.  The base
// b = (1 + m/4) 2^(e-31) is not an E8M0 power of two, so the group's codes
// enter two MFMAs whose E8M0 scales add up to b/4 exactly:
//   m = 0:  1    = 1                 operand B all zero
//   m = 1:  1.25 = 1 + 1/4           B = codes,          scale 2^(e-35)
//   m = 2:  1.5  = 1 + 1/2           B = codes,          scale 2^(e-34)
//   m = 3:  1.75 = 2 - 1/4           B = negated codes,  scale 2^(e-35)
// operand A = codes with scale 2^(e-33), or 2^(e-32) for m = 3.  The E8M0
// byte of 2^k is k + 127.  Byte 0 of the scale word serves operand A, byte 1
// operand B.
__device__ __forceinline__ uint32_t split_scale_word(uint32_t base) {
  const uint32_t e = base >> 2, m = base & 3u;
  const uint32_t sa = e + 94u + (m == 3u ? 1u : 0u);
  const uint32_t sb = e + (m == 2u ? 93u : 92u);
  return sa | (sb << 8);
}

// Stores a lane's operand A (its 24 code bytes) into the operand record at
// rec and operand B into the next record.  A record holds dwords 0..3 of the
// 64 lanes (16 bytes each), then dwords 4..5 (8 bytes each).  The E2M3 sign is
// bit 5 of each 6-bit field.
__device__ __forceinline__ void store_split_operand(uint8_t* rec, int lane, const i6_t& pk, uint32_t base) {
  constexpr uint32_t kSign[3] = {0x20820820u, 0x08208208u, 0x82082082u};   // fields 6s+5, period 96 bits
  const uint32_t m = base & 3u;
  uint32_t wa[6], wb[6];
#pragma unroll
  for (int i = 0; i < 6; ++i) {
    wa[i] = (uint32_t)pk[i];
    wb[i] = m == 0u ? 0u : (m == 3u ? wa[i] ^ kSign[i % 3] : wa[i]);
  }
  *reinterpret_cast<uint4*>(rec + 16 * lane) = make_uint4(wa[0], wa[1], wa[2], wa[3]);
  *reinterpret_cast<uint2*>(rec + 1024 + 8 * lane) = make_uint2(wa[4], wa[5]);
  *reinterpret_cast<uint4*>(rec + kOpRecord + 16 * lane) = make_uint4(wb[0], wb[1], wb[2], wb[3]);
  *reinterpret_cast<uint2*>(rec + kOpRecord + 1024 + 8 * lane) = make_uint2(wb[4], wb[5]);
}

__global__ void __launch_bounds__(512) k_prep_kv_hif4(const half_t* __restrict__ k, const half_t* __restrict__ v,
                                                      const float* __restrict__ s, const int* __restrict__ cu,
                                                      uint8_t* __restrict__ ws, int S, int NB, int heads_kv, int G,
                                                      bool qmean) {
  // workgroup (J, hk, 2b + role): role 0 quantizes K, role 1 V, of block J
  extern __shared__ __align__(16) uint8_t sm[];
  const int J = blockIdx.x, hk = blockIdx.y, b = blockIdx.z >> 1;
  const bool is_v = (blockIdx.z & 1) != 0;
  const int D = 64 * G;
  const int t0 = seq_start(cu, b, S);
  const int L = seq_len(cu, b, S);
  if (64 * J >= L) return;
  const ChunkLayout lay = chunk_layout_hif4(G, qmean);
  uint8_t* chunk = ws + ((size_t)(b * heads_kv + hk) * NB + J) * lay.bytes;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, h = lane >> 5;
  if (!is_v) {
    const int t = wave / G, g = wave % G;
    const int key = 32 * t + (lane & 31);
    const int pos = 64 * J + key;
    // the key's 32 channels 64g + 32h + [0, 32) as 16 fp16 pairs, requested
    // before the smoothing scales are staged so that both loads overlap
    h2_t x[16];
    if (pos < L) {
      typedef uint32_t u4v_t __attribute__((ext_vector_type(4)));
      const u4v_t* src = reinterpret_cast<const u4v_t*>(k + ((size_t)(t0 + pos) * heads_kv + hk) * D + 64 * g + 32 * h);
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) {
        const u4v_t w = src[v4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint32_t wi = w[i];     // copy first: bit-casting an ext_vector element in place misreads it
          x[4 * v4 + i] = __builtin_bit_cast(h2_t, wi);
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i) x[i] = h2_t{(half_t)0, (half_t)0};
    }
    if (s) {
      // this head's smoothing scales and their reciprocals (one division per
      // channel), staged in LDS; then k~ = fp16(k/s) per element
      float* rs = reinterpret_cast<float*>(sm);
      float* ss = rs + D;
      for (int c = threadIdx.x; c < D; c += blockDim.x) {
        const float sc = s[(size_t)hk * D + c];
        ss[c] = sc;
        rs[c] = 1.0f / sc;
      }
      __syncthreads();
      const float* sc = ss + 64 * g + 32 * h;
      const float* rc = rs + 64 * g + 32 * h;
#pragma unroll
      for (int i = 0; i < 16; ++i)
        x[i] = h2_t{div_rn16_rcp((float)x[i][0], sc[2 * i], rc[2 * i]),
                    div_rn16_rcp((float)x[i][1], sc[2 * i + 1], rc[2 * i + 1])};
    }
    if (qmean) {
      // Q-Mean key sums (Algorithm 1's correction term): the exact sum of the
      // key's smoothed channels in float64 (any 256 fp16 values sum exactly),
      // one partial per (32-key half, group) in LDS, then rounded once to fp32.
      double part = 0.0;
#pragma unroll
      for (int i = 0; i < 16; ++i) part += (double)(float)x[i][0] + (double)(float)x[i][1];
      part += __shfl_xor(part, 32);
      double* parts = reinterpret_cast<double*>(sm + 2 * D * sizeof(float));     // [2][G][32]
      if (h == 0) parts[(t * G + g) * 32 + (lane & 31)] = part;
      __syncthreads();
      if (g == 0 && h == 0) {
        double sum = 0.0;
        for (int gg = 0; gg < G; ++gg) sum += parts[(t * G + gg) * 32 + (lane & 31)];
        reinterpret_cast<float*>(chunk + lay.kappa)[32 * t + (lane & 31)] = (float)sum;
      }
    }
    const GroupOps go = rows_quantize(x);
    store_split_operand(chunk + lay.k_op + (size_t)(t * G + g) * 2 * kOpRecord, lane, go.pk, go.base);
    if (h == 0)
      reinterpret_cast<uint32_t*>(chunk + lay.k_scale)[(t * G + g) * 32 + (lane & 31)] = split_scale_word(go.base);
  } else {
    // stage V rows [64J, 64J+64) of this head, zero past the sequence end:
    // 64 * D / 8 pieces of 16 bytes, 4 per thread, all loads issued before
    // the first store (rows past the end load the last row, then store zero)
    half_t* vt = reinterpret_cast<half_t*>(sm);        // [64 keys][D]
    const int pieces_per_row = D / 8;
    uint4 val[4];
    bool live[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = threadIdx.x + r * blockDim.x;
      const int pos = 64 * J + i / pieces_per_row;
      live[r] = pos < L;
      const int row = live[r] ? pos : L - 1;             // L > 64 J >= 0 here
      val[r] = *reinterpret_cast<const uint4*>(v + ((size_t)(t0 + row) * heads_kv + hk) * D +
                                               8 * (i % pieces_per_row));
    }
#pragma unroll
    for (int r = 0; r < 4; ++r)
      reinterpret_cast<uint4*>(vt)[threadIdx.x + r * blockDim.x] = live[r] ? val[r] : make_uint4(0, 0, 0, 0);
    __syncthreads();
    const int dt = wave;
    const int d = 32 * dt + (lane & 31);
    // the lane's 32 keys in the order of the attention kernel's P^ operand:
    // x[t][v2] = keys 32t + 8(v2/2) + 4h + 2(v2%2) + {0, 1} of channel d
    h2_t x[2][8];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int v2 = 0; v2 < 8; ++v2) {
        const int k0 = 32 * t + 8 * (v2 >> 1) + 4 * h + 2 * (v2 & 1);
        x[t][v2] = h2_t{vt[k0 * D + d], vt[(k0 + 1) * D + d]};
      }
    const GroupOps go = keys_quantize(x, lane, h);
    store_split_operand(chunk + lay.v_op + (size_t)dt * 2 * kOpRecord, lane, go.pk, go.base);
    if (h == 0) reinterpret_cast<uint32_t*>(chunk + lay.v_scale)[d] = split_scale_word(go.base);
  }
}

// ---------------------------------------------------------------------------
// Attention pre-pass (FP16 operands, the C16V16 reference).  Same chunking;
//   K operand [2][D/16][64 lanes][8 halves]: lane l holds key 32t + l%32,
//     channels 16kc + 8(l/32) + [0,8) -- A operand of the 32x32x16 f16 MFMA;
//   V operand [D/32][4 chunks][64 lanes][8 halves]: lane l holds channel
//     32dt + l%32 and, at slot e of key chunk c = 2t + jp, the key
//     32t + 8(2jp + e/4) + 4(l/32) + e%4.
__global__ void __launch_bounds__(256) k_prep_kv_fp16(const half_t* __restrict__ k, const half_t* __restrict__ v,
                                                      const int* __restrict__ cu, uint8_t* __restrict__ ws, int S,
                                                      int NB, int heads_kv, int D) {
  const int J = blockIdx.x, hk = blockIdx.y, b = blockIdx.z;
  const int t0 = seq_start(cu, b, S);
  const int L = seq_len(cu, b, S);
  if (64 * J >= L) return;
  const ChunkLayout lay = chunk_layout_fp16(D);
  uint8_t* chunk = ws + ((size_t)(b * heads_kv + hk) * NB + J) * lay.bytes;
  const int lane = threadIdx.x & 63, h = lane >> 5;
  // K: items (t, kc, lane)
  const int nk = 2 * (D / 16) * 64;
  for (int it = threadIdx.x; it < nk; it += blockDim.x) {
    const int ln = it & 63, kc = (it >> 6) % (D / 16), t = (it >> 6) / (D / 16);
    const int pos = 64 * J + 32 * t + (ln & 31);
    uint4 val = make_uint4(0, 0, 0, 0);
    if (pos < L)
      val = *reinterpret_cast<const uint4*>(k + ((size_t)(t0 + pos) * heads_kv + hk) * D + 16 * kc + 8 * (ln >> 5));
    reinterpret_cast<uint4*>(chunk + lay.k_op)[it] = val;
  }
  // V: items (dt, c, lane)
  const int nv = (D / 32) * 4 * 64;
  for (int it = threadIdx.x; it < nv; it += blockDim.x) {
    const int ln = it & 63, c = (it >> 6) & 3, dt = (it >> 8);
    const int hh = ln >> 5, d = 32 * dt + (ln & 31);
    const int t = c >> 1, jp = c & 1;
    h8_t val;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int pos = 64 * J + 32 * t + 8 * (2 * jp + (e >> 2)) + 4 * hh + (e & 3);
      val[e] = pos < L ? v[((size_t)(t0 + pos) * heads_kv + hk) * D + d] : (half_t)0.0f;
    }
    reinterpret_cast<h8_t*>(chunk + lay.v_op)[it] = val;
  }
  (void)h;
}

// ---------------------------------------------------------------------------
// Calibration reductions.  stats layout: [n][2][Hkv][D] uint32 holding the
// bits of non-negative floats (order-preserving): index 0 = max|K|, 1 = max|Q|
// (over the query heads of the group).  hist: 32768 uint64 bins of the fp16
// magnitude bit pattern of every K element.
__global__ void k_fill_u32(uint32_t* __restrict__ p, size_t n, uint32_t val) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = val;
}

__global__ void __launch_bounds__(256) k_calib_absmax(const half_t* __restrict__ x, uint32_t* __restrict__ stats,
                                                      int S, int heads, int heads_kv, int D, int which) {
  // grid: (token chunks, n); each thread handles one channel pair over a
  // slice of tokens for every head.
  const int n = blockIdx.y;
  const int rows_per_block = 64;
  const int r0 = blockIdx.x * rows_per_block;
  const int cols = heads * D;
  const half_t* base = x + (size_t)n * S * cols;
  uint32_t* st = stats + ((size_t)n * 2 + which) * heads_kv * D;
  const int grp = heads / heads_kv;
  for (int c = threadIdx.x; c < cols; c += blockDim.x) {
    float m = 0.0f;
    for (int r = r0; r < min(r0 + rows_per_block, S); ++r) m = fmaxf(m, fabsf((float)base[(size_t)r * cols + c]));
    const int hh = c / D, d = c % D;
    atomicMax(&st[(size_t)(hh / grp) * D + d], __float_as_uint(m));
  }
}

// Per-workgroup LDS histogram with two 16-bit counters per word; the host
// sizes the grid so that no workgroup sees more than 32768 elements, which
// keeps every counter below 2^16.
__global__ void __launch_bounds__(1024) k_calib_hist(const half_t* __restrict__ k, size_t n, size_t per_block,
                                                     unsigned long long* __restrict__ hist) {
  __shared__ uint32_t lh[16384];
  for (int i = threadIdx.x; i < 16384; i += blockDim.x) lh[i] = 0;
  __syncthreads();
  const uint16_t* kb = reinterpret_cast<const uint16_t*>(k);
  const size_t i0 = (size_t)blockIdx.x * per_block;
  const size_t i1 = i0 + per_block < n ? i0 + per_block : n;
  for (size_t i = i0 + threadIdx.x; i < i1; i += blockDim.x) {
    const uint32_t bin = kb[i] & 0x7FFFu;
    atomicAdd(&lh[bin >> 1], 1u << (16 * (bin & 1u)));
  }
  __syncthreads();
  for (int i = threadIdx.x; i < 16384; i += blockDim.x) {
    const uint32_t w = lh[i];
    if (w & 0xFFFFu) atomicAdd(&hist[2 * i], (unsigned long long)(w & 0xFFFFu));
    if (w >> 16) atomicAdd(&hist[2 * i + 1], (unsigned long long)(w >> 16));
  }
}

// ---------------------------------------------------------------------------
// Pairs of inputs go through the packed routine the attention kernels use.
__global__ void k_selftest_exp2(const half_t* __restrict__ x, half_t* __restrict__ y, long n) {
  const long i = 2 * ((long)blockIdx.x * blockDim.x + threadIdx.x);
  if (i >= n) return;
  h2_t v = {x[i], i + 1 < n ? x[i + 1] : (half_t)0.0f};
  const h2_t r = exp2_h2(v);
  y[i] = r[0];
  if (i + 1 < n) y[i + 1] = r[1];
}

// ---------------------------------------------------------------------------
// Host launchers.
hipError_t launch_quant_rows(const half_t* x, const float* s, uint8_t* codes, uint32_t* meta, long n_rows,
                             int heads, int heads_kv, int D, bool is_k, hipStream_t st) {
  const int G = D / 64;
  const long n_groups = n_rows * heads * G;
  if (n_groups == 0) return hipSuccess;
  const int waves = 4;
  const long blocks = (n_groups + 32 * waves - 1) / (32 * waves);
  if (is_k)
    k_quant_rows<true><<<dim3((unsigned)blocks), dim3(64 * waves), 0, st>>>(x, s, codes, meta, (int)n_groups, heads,
                                                                            heads_kv, G);
  else
    k_quant_rows<false><<<dim3((unsigned)blocks), dim3(64 * waves), 0, st>>>(x, s, codes, meta, (int)n_groups, heads,
                                                                             heads_kv, G);
  return hipGetLastError();
}

hipError_t launch_quant_v(const half_t* v, const int* cu, uint8_t* codes, uint32_t* meta, int batch, int S, int NB,
                          int heads_kv, int D, hipStream_t st) {
  const long n_groups = (long)batch * NB * heads_kv * D;
  if (n_groups == 0) return hipSuccess;
  const long blocks = (n_groups + 127) / 128;
  k_quant_v_canon<<<dim3((unsigned)blocks), dim3(256), 0, st>>>(v, cu, codes, meta, batch, S, NB, heads_kv, D);
  return hipGetLastError();
}

hipError_t launch_prep_kv(const half_t* k, const half_t* v, const float* s, const int* cu, uint8_t* ws, int batch,
                          int S, int NB, int heads_kv, int D, bool fp16, bool qmean, hipStream_t st) {
  dim3 grid(NB, heads_kv, batch);
  if (fp16)
    k_prep_kv_fp16<<<grid, dim3(256), 0, st>>>(k, v, cu, ws, S, NB, heads_kv, D);
  else
    k_prep_kv_hif4<<<dim3(NB, heads_kv, 2 * batch), dim3(64 * 2 * (D / 64)), 64 * D * sizeof(half_t), st>>>(
        k, v, s, cu, ws, S, NB, heads_kv, D / 64, qmean);
  return hipGetLastError();
}

hipError_t launch_calib(const half_t* q, const half_t* k, int n, int S, int hq, int hkv, int D, uint32_t* stats,
                        unsigned long long* hist, hipStream_t st) {
  const size_t n_stats = (size_t)n * 2 * hkv * D;
  k_fill_u32<<<dim3(256), dim3(256), 0, st>>>(stats, n_stats, 0u);
  k_fill_u32<<<dim3(64), dim3(256), 0, st>>>(reinterpret_cast<uint32_t*>(hist), 2 * 32768, 0u);
  dim3 grid((S + 63) / 64, n);
  k_calib_absmax<<<grid, dim3(256), 0, st>>>(k, stats, S, hkv, hkv, D, 0);
  k_calib_absmax<<<grid, dim3(256), 0, st>>>(q, stats, S, hq, hkv, D, 1);
  const size_t nk = (size_t)n * S * hkv * D;
  const size_t per_block = 32768;
  const size_t nblk = (nk + per_block - 1) / per_block;
  if (nblk > 0) k_calib_hist<<<dim3((unsigned)nblk), dim3(1024), 0, st>>>(k, nk, per_block, hist);
  return hipGetLastError();
}

hipError_t launch_selftest_exp2(const half_t* x, half_t* y, long n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  k_selftest_exp2<<<dim3((unsigned)((n + 511) / 512)), dim3(256), 0, st>>>(x, y, n);
  return hipGetLastError();
}

}  // namespace hifa4
