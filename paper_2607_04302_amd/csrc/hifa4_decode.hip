// HiFA4 decode step on a packed HIF4 K/V cache (gfx950).
//
// Paper: Algorithm 1 for one query row per sequence (the newest token, which
// sees every cached key) with Section 4.5's P-Reordering; the cache holds K^
// and V^ in the packed 4.5-bit HIF4 format of the Background's HIF4
// paragraph.  The paper leaves decode and the KV-cache footprint open.
//
// The cache is the canonical layout (hifa4_quantize_qk, hifa4_quantize_v):
// per group 32 bytes of sign-magnitude nibbles and one metadata word.  One
// decode row has too little work per sequence for one workgroup, so the key
// range is split; the split must not change any P^ code, because P^ depends
// on the running maximum entering each 64-key block.  Three kernels keep every
// decision of the sequential loop (where the splits alone fill the chip, the
// first two are one kernel: see "1+2" below):
//   1. scores: per (sequence, run of 64-key blocks, kv head) the query rows
//      of the GQA group are smoothed and quantized (Q^ = HIF4(fp16(q s))),
//      then the fp16 scores S2 are stored with each row's block maximum;
//   2. splits: each wave takes a run of blocks and starts from the running
//      maximum the sequential loop has at its first block (the prefix maximum
//      of the stored block maxima), then applies the FP16 softmax,
//      P^ = HIF4(P) and the PV product as the sequential loop does; it writes
//      its partial O_s and l_s, both relative to the running maximum at its
//      last block;
//   3. merge: O = sum_s O_s R_s and l = sum_s l_s R_s, where R_s is the product
//      of the rescale factors r_J = E(fp16(m_{J-1} - m_J)) of all blocks after
//      split s: the sequential recurrence O <- r_J O + P^_J V^_J unrolled.
//
// Both contractions run on the int8 MFMA (32x32x32, int32 accumulate).  A HIF4
// element is +-u 2^-sh times b/4 (u <= 7, sh <= 2), so 4 u 2^-sh = +-u << (2-sh)
// is an integer in [-28, 28]: the group's codes become int8 operands with two
// shifts and a sign fix per four elements, every 64-element dot product is
// exact in int32, and the bases (E6M2, three significant bits) are applied
// in an fp32 epilogue where every product stays exact.  The scores therefore
// follow the library's score contract bit for bit, and the PV partial sums of
// a block are exact before the fp32 rescale-and-add.
//
// MFMA operand convention: lane l holds row / column (l & 31) of A / B and
// sixteen k indices chosen by the half h = l >> 5; a 64-element group is two
// MFMAs, the first over the group's quarters 2h (bytes 16h..16h+7), the
// second over quarters 2h+1 (bytes 16h+8..16h+15), so each lane reads 16
// contiguous code bytes.  Only the pairing of k indices between A and B
// matters for a dot product, and both operands place a quarter's sixteen
// elements in the same (decode) order.  The output lane l holds column
// (l & 31) and, in its first four values, rows 4h + c, so a wave serves at
// most eight query rows: GQA groups of up to 8 heads per kv head.
//
// Workgroups hold one wave per kv head (up to eight): the heads of a token
// share cache lines, so the lines are read once by one compute unit.
#include <atomic>
#include <random>

#include "hifa4_device.h"
#include "hifa4_decode.h"
#include "hifa4_internal.h"
#include "hifa4_packed.h"

namespace hifa4 {

namespace {

typedef int i4_t __attribute__((ext_vector_type(4)));
typedef int i16_t __attribute__((ext_vector_type(16)));
typedef unsigned short u16x2_t __attribute__((ext_vector_type(2)));

// Blocks per score wave: 8 when that still gives at least two workgroups per
// compute unit, else 2, else 1 (short or single sequences).  Blocks per split:
// the longest of 8, 4 and 2 that gives a workgroup per compute unit, with at
// most 128 splits per row, since every split also pays a prefix maximum over
// the blocks before it, a partial output in fp32 and its share of the merge.
constexpr int kScoreRuns[3] = {8, 2, 1};
constexpr int kSplitLengths[3] = {8, 4, 2};
constexpr int kMinScoreWorkgroups = 512;
constexpr int kMinSplitWorkgroups = 256;
constexpr int kMaxSplitsPerRow = 128;
constexpr int kMaxWaves = 8;             // kv heads per workgroup

__device__ __forceinline__ int dseq_start(const int* cu, int b, int S) { return cu ? cu[b] : b * S; }
// a length above max_seqlen is outside the contract; clamping it keeps every
// access inside the caller's buffers
__device__ __forceinline__ int dseq_len(const int* cu, int b, int S) { return cu ? min(cu[b + 1] - cu[b], S) : S; }

__device__ __forceinline__ half_t exp2_h(half_t x) { return exp2_h2(h2_t{x, (half_t)0})[0]; }
__device__ __forceinline__ half_t hmax(half_t a, half_t b) { return a > b ? a : b; }

// Shift amounts 2 - sh of the two E3 blocks of each of the words 2Q and 2Q+1
// of a group (elements 16Q..16Q+15), packed as 16-bit halves: low half =
// first four elements of the word, high half = last four.
__device__ __forceinline__ void quarter_shifts(uint32_t meta, int Q, uint32_t& k0, uint32_t& k1) {
  const uint32_t e2 = (meta >> (8 + 2 * Q)) & 3u;        // E2 of words 2Q, 2Q+1
  const uint32_t e3 = (meta >> (16 + 4 * Q)) & 15u;      // E3 of blocks 4Q..4Q+3
  const uint32_t a0 = e2 & 1u, a1 = e2 >> 1;
  k0 = (2u - a0 - (e3 & 1u)) | ((2u - a0 - ((e3 >> 1) & 1u)) << 16);
  k1 = (2u - a1 - ((e3 >> 2) & 1u)) | ((2u - a1 - (e3 >> 3)) << 16);
}

// Four sign-magnitude elements, one per byte (magnitude in `mag`, sign bit in
// bit 0 of each byte of `sgn`), to int8 +-mag << k with k per 16-bit half.
// The magnitudes stay below 32 after the shift, so no byte spills into the
// next; a zero magnitude never carries a sign (zero is stored as +0).
__device__ __forceinline__ uint32_t to_i8x4(uint32_t mag, uint32_t sgn, uint32_t k) {
  const u16x2_t v = __builtin_bit_cast(u16x2_t, mag) << __builtin_bit_cast(u16x2_t, k);
  const uint32_t m = __builtin_bit_cast(uint32_t, v);
  const uint32_t neg = (sgn << 8) - sgn;                 // 0xff in every negative byte
  return (m ^ neg) + sgn;                                // per-byte two's complement
}

// Sixteen elements (the 8 code bytes w of quarter Q of a group) as int8
// operands 4 * (+-u 2^-sh).  Byte order: register 0 = elements 0,2,4,6,
// register 1 = 1,3,5,7, register 2 = 8,10,12,14, register 3 = 9,11,13,15
// (relative to 16Q).
__device__ __forceinline__ i4_t decode_quarter(uint32_t wx, uint32_t wy, uint32_t meta, int Q) {
  uint32_t k0, k1;
  quarter_shifts(meta, Q, k0, k1);
  i4_t r;
  r[0] = (int)to_i8x4(wx & 0x07070707u, (wx >> 3) & 0x01010101u, k0);
  r[1] = (int)to_i8x4((wx >> 4) & 0x07070707u, (wx >> 7) & 0x01010101u, k0);
  r[2] = (int)to_i8x4(wy & 0x07070707u, (wy >> 3) & 0x01010101u, k1);
  r[3] = (int)to_i8x4((wy >> 4) & 0x07070707u, (wy >> 7) & 0x01010101u, k1);
  return r;
}

// Byte index, inside the 16-byte operand of a quarter, of its element e
// (0..15) in the order decode_quarter produces.
__device__ __forceinline__ constexpr int operand_byte(int e) {
  return 4 * (2 * (e >> 3) + (e & 1)) + ((e & 7) >> 1);
}

// Exact int32 dot products of a whole 64-element group: the MFMA over the
// lane's first quarter, then the second, accumulated.
__device__ __forceinline__ i16_t group_dot(i4_t a0, i4_t a1, uint4 w, uint32_t meta, int h) {
  const i16_t z = {};
  const i16_t c = __builtin_amdgcn_mfma_i32_32x32x32_i8(a0, decode_quarter(w.x, w.y, meta, 2 * h), z, 0, 0, 0);
  return __builtin_amdgcn_mfma_i32_32x32x32_i8(a1, decode_quarter(w.z, w.w, meta, 2 * h + 1), c, 0, 0, 0);
}

struct DecodeArgs {
  const half_t* q;         // raw decode queries [batch, Hq, D] fp16
  const float* s;          // smoothing scales [Hkv, D] or null
  const uint8_t* kc;       // canonical K^ cache [tokens, Hkv, G, 32]
  const uint32_t* km;      // [tokens, Hkv, G]
  const uint8_t* vc;       // canonical V^ cache [batch, NB, Hkv, D, 32]
  const uint32_t* vm;      // [batch, NB, Hkv, D]
  const int* cu;
  half_t* s2;              // scores [batch, Hq, NB, 64]
  half_t* mx;              // block maxima [batch, Hq, mxs]
  float* opart;            // [batch, Hq, n_split, D]
  float4* spart;           // [batch, Hq, n_split]: l, product of the split's
                           // rescale factors, running max after its last block
  half_t* o;               // [batch, Hq, D]
  float* lse;              // [Hq, batch]
  uint8_t* dbg_codes;      // [Hq, batch, NB, 32] or null
  uint32_t* dbg_meta;      // [Hq, batch, NB]
  int batch, S, NB, hq, hkv, D, n_split, waves, bps;
  int mxs;                 // row stride of the block maxima: NB rounded up to 8
  float c;
  uint64_t* runmax;        // fused path: [batch, Hq, n_split] run maxima, epoch-tagged;
                           // the merge kernel clears each row's words after the splits
  uint32_t epoch;          // fused path: this call's tag (never 0)
  int spin_limit;          // polls before a look-back wait gives up
  int publish;             // 0: the fused kernel publishes no run maxima (testing the give-up)
};

// One wave's share of a workgroup: kv head hk of sequence b, blocks
// [J0, J1) of run (or split) `part`.
struct WaveSpan {
  int hk, b, L, J0, J1, t0, grp, part;
  size_t row0;             // first query row of the GQA group
};

// False when the wave has nothing to do (no kv head, or no block in range).
__device__ __forceinline__ bool wave_span(const DecodeArgs& a, int blocks, WaveSpan& w) {
  w.hk = blockIdx.x * a.waves + (int)(threadIdx.x >> 6);
  if (w.hk >= a.hkv) return false;
  w.b = blockIdx.z;
  w.part = blockIdx.y;
  w.L = dseq_len(a.cu, w.b, a.S);
  const int nblk = (w.L + 63) >> 6;
  w.J0 = w.part * blocks;
  if (w.J0 >= nblk) return false;
  w.J1 = min(w.J0 + blocks, nblk);
  w.t0 = dseq_start(a.cu, w.b, a.S);
  w.grp = a.hq / a.hkv;
  w.row0 = (size_t)w.b * a.hq + (size_t)w.hk * w.grp;
  return true;
}

// LDS of the score phase, per wave: the run's scores [row][block][key], the
// block maxima, Q^'s A operands [row][group][64] and their bases.
template <int G, int RUN>
struct ScoreLds {
  half_t s[kMaxWaves][8][RUN * 64];
  half_t m[kMaxWaves][8][RUN];
  alignas(16) int8_t q[kMaxWaves][8 * G * 64];
  uint32_t qb[kMaxWaves][8 * G];
};

// ---------------------------------------------------------------------------
// 1. Scores and block maxima.  Wave = kv head, workgroup = (kv heads, run of
// blocks, sequence).  A = the GQA group's query rows (rows >= the group size
// are zero), B = 32 keys of the block; per (32-key tile, channel group) the
// two MFMAs give the exact group dots 16 * sum(q_unit * k_unit) of query rows
// 4h + c with key (l & 31) of the tile.  Epilogue per group: d_g = dot * b_K/64
// (exact), the group's exact term t_g = d_g * b_Q,g/4, the terms summed in
// order in fp32 (a fused multiply-add of the exact product rounds exactly the
// sum), S2 = fp16(fp32(sum * c)).  Two register buffers in fixed
// roles keep the next two blocks' codes in flight; the scores and maxima of
// the run are collected in LDS and stored after the last block, so the loop
// issues loads only.
template <int G, int RUN>
__device__ __forceinline__ void score_run(const DecodeArgs& a, const WaveSpan& w, ScoreLds<G, RUN>& sl) {
  constexpr int kScoreBlocksPerWave = RUN;
  const int wave = (int)(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, n = lane & 31, h = lane >> 5;
  const int hk = w.hk, L = w.L, J0 = w.J0, J1 = w.J1, t0 = w.t0, grp = w.grp;
  const size_t row0 = w.row0;
  struct KBlock {
    uint4 w[2][G];
    uint32_t meta[2][G];
  };
  auto load = [&](int J, KBlock& kb) {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int key = 64 * J + 32 * t + n;
      const int kk = key < L ? key : L - 1;                  // rows past the end are masked below
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const size_t gi = ((size_t)(t0 + kk) * a.hkv + hk) * G + g;
        kb.w[t][g] = *reinterpret_cast<const uint4*>(a.kc + gi * 32 + 16 * h);
        kb.meta[t][g] = a.km[gi];
      }
    }
  };
  // Q^ of the group's query rows, quantized here (each workgroup of the
  // sequence repeats it: a few hundred instructions against a separate
  // launch).  Pass p: lane i takes (row, group) pair 4p + (i >> 4) and its
  // channels 4(i & 15)..+3, one E3 block; q~ = fp16(fp32(q) * s).  Every load
  // of every pass is issued first (rows past the group read row 0).
  constexpr int D = 64 * G;
  constexpr int kQPasses = 2 * G;                           // 8 rows x G groups / 4 per pass
  const int kq = lane & 15;
  uint2 qraw[kQPasses];
  float4 qs[kQPasses];
#pragma unroll
  for (int p = 0; p < kQPasses; ++p) {
    const int pi = 4 * p + (lane >> 4), r = pi / G, g = pi % G;
    const int ch = 64 * g + 4 * kq;
    qraw[p] = *reinterpret_cast<const uint2*>(a.q + (row0 + (r < grp ? r : 0)) * D + ch);
    qs[p] = a.s ? *reinterpret_cast<const float4*>(a.s + (size_t)hk * D + ch) : make_float4(1.0f, 1.0f, 1.0f, 1.0f);
  }
  // every prefetch is unconditional (past the run's end it reloads the last
  // block), so the number of loads in flight is the same on every path
  KBlock b0, b1;
  load(J0, b0);
  // HIF4 of each group (the row base over 16 lanes, E2 over a lane pair, E3
  // in-lane), the int8 operand values 4u 2^-sh with their signs written to
  // LDS in the A-operand layout, the bases beside them
  int8_t* lq = sl.q[wave];
#pragma unroll
  for (int p = 0; p < kQPasses; ++p) {
    const int pi = 4 * p + (lane >> 4), r = pi / G, g = pi % G;
    if (4 * p >= grp * G) break;                             // uniform: no pair of this pass is live
    // q~ = fp16(q * s), the exact product rounded once (mixed-precision fma)
    const h2_t y01 = smooth_mul2(__builtin_bit_cast(h2_t, qraw[p].x), qs[p].x, qs[p].y);
    const h2_t y23 = smooth_mul2(__builtin_bit_cast(h2_t, qraw[p].y), qs[p].z, qs[p].w);
    const half_t xsm[4] = {y01[0], y01[1], y23[0], y23[1]};
    float ax[4];
    bool neg[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      ax[j] = fabsf((float)xsm[j]);
      neg[j] = (float)xsm[j] < 0.0f;
    }
    const float a4 = fmaxf(fmaxf(ax[0], ax[1]), fmaxf(ax[2], ax[3]));
    const float a8 = fmaxf(a4, __shfl_xor(a4, 1));
    float A = a8;
#pragma unroll
    for (int o = 2; o < 16; o <<= 1) A = fmaxf(A, __shfl_xor(A, o));
    const uint32_t base = e6m2_ceil(A);
    const float bval = e6m2_value(base);
    const bool e2 = a8 <= 0.875f * bval;
    const bool e3 = a4 <= (e2 ? 0.4375f : 0.875f) * bval;
    const int sh = (int)e2 + (int)e3;
    const float R = hif4_rcp_step(base);
    const float C = round_const(sh);
    if (r < grp) {
      int8_t* dst = lq + (r * G + g) * 64 + 16 * (kq >> 2);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int u = (int)(__float_as_uint(__builtin_fmaf(ax[j], R, C)) - __float_as_uint(C));
        const int v = u << (2 - sh);
        dst[operand_byte(4 * (kq & 3) + j)] = (int8_t)(neg[j] ? -v : v);
      }
      if (kq == 0) sl.qb[wave][r * G + g] = base;
    }
  }
  // A operands of row n (zero past the group), weights of the output rows 4h + c
  i4_t qa[G][2];
  float wq[G][4];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    qa[g][0] = qa[g][1] = i4_t{0, 0, 0, 0};
    if (n < grp) {
      qa[g][0] = *reinterpret_cast<const i4_t*>(lq + (n * G + g) * 64 + 32 * h);
      qa[g][1] = *reinterpret_cast<const i4_t*>(lq + (n * G + g) * 64 + 32 * h + 16);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int r = 4 * h + c;
      wq[g][c] = 0.25f * e6m2_value(sl.qb[wave][(r < grp ? r : 0) * G + g]);
    }
  }
  load(min(J0 + 1, J1 - 1), b1);
  half_t* ls = &sl.s[wave][0][0];
  auto compute = [&](const KBlock& kb, int i) {
    const int J = J0 + i;
    float acc[2][4];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const uint32_t meta = kb.meta[t][g];
        const i16_t dot = group_dot(qa[g][0], qa[g][1], kb.w[t][g], meta, h);
        const float bk = e6m2_value(meta & 255u) * 0.015625f;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const float d = (float)dot[c] * bk;                      // exact
          acc[t][c] = g == 0 ? d * wq[0][c] : __builtin_fmaf(d, wq[g][c], acc[t][c]);
        }
      }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int r = 4 * h + c;
      half_t sv[2];
      float m = -__builtin_inff();
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        sv[t] = 64 * J + 32 * t + n < L ? (half_t)(acc[t][c] * a.c) : (half_t)(-__builtin_inff());
        m = fmaxf(m, (float)sv[t]);
      }
#pragma unroll
      for (int o = 1; o < 32; o <<= 1) m = fmaxf(m, __shfl_xor(m, o));
      if (r < grp) {
        ls[r * (kScoreBlocksPerWave * 64) + 64 * i + n] = sv[0];
        ls[r * (kScoreBlocksPerWave * 64) + 64 * i + 32 + n] = sv[1];
        if (n == 0) sl.m[wave][r][i] = (half_t)m;
      }
    }
  };
#pragma unroll
  for (int i = 0; i < kScoreBlocksPerWave; i += 2) {
    if (J0 + i < J1) compute(b0, i);
    if (i + 2 < kScoreBlocksPerWave) load(min(J0 + i + 2, J1 - 1), b0);
    if (i + 1 < kScoreBlocksPerWave && J0 + i + 1 < J1) compute(b1, i + 1);
    if (i + 3 < kScoreBlocksPerWave) load(min(J0 + i + 3, J1 - 1), b1);
  }
}

template <int G, int RUN>
__global__ void __launch_bounds__(64 * kMaxWaves, (G <= 2 ? 4 : 2)) k_decode_scores(DecodeArgs a) {
  __shared__ __align__(16) ScoreLds<G, RUN> sl;
  WaveSpan w;
  if (!wave_span(a, RUN, w)) return;
  score_run<G, RUN>(a, w, sl);
  // the run's scores (J1 - J0 blocks of 64, contiguous per row) and maxima
  const int wave = (int)(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int nb = w.J1 - w.J0;
  for (int r = 0; r < w.grp; ++r) {
    const uint2* src = reinterpret_cast<const uint2*>(&sl.s[wave][r][0]);
    uint2* dst = reinterpret_cast<uint2*>(a.s2 + ((w.row0 + r) * a.NB + w.J0) * 64);
    for (int k = lane; k < nb * 16; k += 64) dst[k] = src[k];
    if (lane < nb) a.mx[(w.row0 + r) * a.mxs + w.J0 + lane] = sl.m[wave][r][lane];
  }
}

// ---------------------------------------------------------------------------
// 2. Splits.  Wave = kv head, workgroup = (kv heads, split, sequence).  Per
// block, the FP16 softmax and P^ = HIF4(P) run on every lane: lane i takes
// query row 4p + (i >> 4) (pass p < RP) and its keys 4(i & 15)..+3, one E3
// block; E2 pairs two lanes, the row base sixteen.  The int8 values
// 4 u 2^-sh go to LDS in the A-operand layout (row, quarter, decode order),
// from where lane (row l & 31, half h) reads its two operands.  B = 32
// channels of the block's V^ groups; per 32-channel tile the two MFMAs give
// the exact block sums, and O[row][ch] = fma(O, r_row, dot * b_V/16 * b_P/16).
constexpr int kLookBatch = 4;                    // run maxima per lane per round
constexpr int kSpinLimit = 1 << 20;

// The running maximum entering run w.part of the lane's softmax row (pass
// p): the maximum of the earlier runs' epoch-tagged maxima of the sequence,
// 16 lanes per row, kLookBatch words each per round, every load of a round
// in flight before the first is checked.  A spin limit ends every wait; a
// wait that gives up sets `lost` (the split then poisons its partial, so the
// row's O and LSE come out NaN instead of silently wrong).
__device__ __forceinline__ float look_back(const DecodeArgs& a, const WaveSpan& w, int row, bool& lost) {
  const int kq = threadIdx.x & 15;
  const uint64_t* f = a.runmax + (w.row0 + row) * a.n_split;
  float mm = -__builtin_inff();
  lost = false;
  for (int q0 = 0; q0 < w.part; q0 += 16 * kLookBatch) {
    uint64_t wd[kLookBatch];
#pragma unroll
    for (int k = 0; k < kLookBatch; ++k) {
      const int q = q0 + 16 * k + kq;
      wd[k] = q < w.part ? __hip_atomic_load(f + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0;
    }
#pragma unroll
    for (int k = 0; k < kLookBatch; ++k) {
      const int q = q0 + 16 * k + kq;
      if (q < w.part) {
        uint64_t v = wd[k];
        for (int it = 0; (uint32_t)(v >> 32) != a.epoch && it < a.spin_limit; ++it) {
          __builtin_amdgcn_s_sleep(2);
          v = __hip_atomic_load(f + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if ((uint32_t)(v >> 32) == a.epoch) mm = fmaxf(mm, (float)__builtin_bit_cast(half_t, (uint16_t)v));
        else lost = true;
      }
    }
  }
  return mm;
}

// FROM_LDS: the scores and block maxima of the split's blocks are in this
// wave's LDS (lsc [8 rows][BPS * 64], lmx [8 rows][BPS]) and the running
// maximum entering the split comes from the earlier runs' published maxima
// (look_back, once the first V^ blocks are in flight); otherwise all of it
// comes from HBM.
template <int NT, int RP, int NORM, bool DEBUG, int BPS, bool FROM_LDS>
__device__ __forceinline__ void split_run(const DecodeArgs& a, const WaveSpan& w, uint8_t* lp, const half_t* lsc,
                                          const half_t* lmx) {
  constexpr int kBlocksPerSplit = BPS;
  constexpr int D = 32 * NT;
  const int lane = threadIdx.x & 63, n = lane & 31, h = lane >> 5;
  const int hk = w.hk, b = w.b, sp = w.part, J0 = w.J0, J1 = w.J1, grp = w.grp;
  const size_t row0 = w.row0;
  const int kq = lane & 15;                      // keys 4kq..4kq+3 of the block
  const int quarter = kq >> 2;                   // their group quarter
  int prow[RP];                                  // softmax row of this lane per pass
#pragma unroll
  for (int p = 0; p < RP; ++p) {
    const int r = 4 * p + (lane >> 4);
    prow[p] = r < grp ? r : 0;
  }
  struct VBlock {
    uint4 w[NT];
    uint32_t meta[NT];
    uint2 s[RP];
    half_t mx[RP];
  };
  auto load = [&](int J, VBlock& vb) {
    const size_t vg = (((size_t)b * a.NB + J) * a.hkv + hk) * D;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const size_t gi = vg + 32 * t + n;
      vb.w[t] = *reinterpret_cast<const uint4*>(a.vc + gi * 32 + 16 * h);
      vb.meta[t] = a.vm[gi];
    }
    if constexpr (!FROM_LDS) {
#pragma unroll
      for (int p = 0; p < RP; ++p) {
        const size_t rj = (row0 + prow[p]) * a.NB + J;
        vb.s[p] = *reinterpret_cast<const uint2*>(a.s2 + rj * 64 + 4 * kq);
        vb.mx[p] = a.mx[(row0 + prow[p]) * a.mxs + J];
      }
    }
  };
  // every prefetch is unconditional (past the split's end it reloads the last
  // block), so the number of loads in flight is the same on every path
  VBlock b0, b1;
  load(J0, b0);
  load(min(J0 + 1, J1 - 1), b1);
  // the running maximum entering block J0 of each softmax row: the prefix
  // maximum of the row's block maxima.  The 16 lanes of a row read 8 maxima
  // per load; every load of a round is issued before the first is used.
  constexpr int kPrefixLoads = 4 / RP;
  half_t m[RP];
  float l[RP], prod[RP];
  h2_t pm[RP];
#pragma unroll
  for (int p = 0; p < RP; ++p) {
    l[p] = 0.0f;
    prod[p] = 1.0f;
    pm[p] = h2_t{(half_t)(-__builtin_inff()), (half_t)(-__builtin_inff())};
  }
  const int nch = FROM_LDS ? 0 : (J0 + 7) >> 3;  // chunks of 8 maxima before J0
  for (int c0 = 0; c0 < nch; c0 += 16 * kPrefixLoads) {
    uint4 w[RP][kPrefixLoads];
    int nv[kPrefixLoads];
#pragma unroll
    for (int k = 0; k < kPrefixLoads; ++k) {
      const int c = c0 + 16 * k + kq;
      const int ce = c < nch ? c : 0;            // past the end: chunk 0 again (max is idempotent)
      nv[k] = J0 - 8 * ce;                       // maxima of the chunk before J0
#pragma unroll
      for (int p = 0; p < RP; ++p)
        w[p][k] = *reinterpret_cast<const uint4*>(a.mx + (row0 + prow[p]) * a.mxs + 8 * ce);
    }
#pragma unroll
    for (int k = 0; k < kPrefixLoads; ++k)
#pragma unroll
      for (int p = 0; p < RP; ++p) {
        const uint32_t x[4] = {w[p][k].x, w[p][k].y, w[p][k].z, w[p][k].w};
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          uint32_t v = x[d];
          if (2 * d + 1 >= nv[k]) v = (v & 0xFFFFu) | 0xFC000000u;     // -inf
          if (2 * d >= nv[k]) v = 0xFC00FC00u;
          pm[p] = hmax2(pm[p], __builtin_bit_cast(h2_t, v));
        }
      }
  }
  bool lost[RP];                                 // a look-back wait of the row gave up
#pragma unroll
  for (int p = 0; p < RP; ++p) {
    bool lp_ = false;
    float mm = FROM_LDS ? look_back(a, w, prow[p], lp_) : fmaxf((float)pm[p][0], (float)pm[p][1]);
    int lf = lp_ ? 1 : 0;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      mm = fmaxf(mm, __shfl_xor(mm, o));
      lf |= __shfl_xor(lf, o);
    }
    m[p] = (half_t)mm;
    lost[p] = lf != 0;
  }
  float O[NT][4];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int c = 0; c < 4; ++c) O[t][c] = 0.0f;
  auto block = [&](const VBlock& cur, int J) {
    float rr[RP], sp16[RP];
#pragma unroll
    for (int p = 0; p < RP; ++p) {
      const int r = 4 * p + (lane >> 4);
      uint2 s4;
      half_t bmax;
      if constexpr (FROM_LDS) {
        s4 = *reinterpret_cast<const uint2*>(lsc + prow[p] * (BPS * 64) + 64 * (J - J0) + 4 * kq);
        bmax = lmx[prow[p] * BPS + (J - J0)];
      } else {
        s4 = cur.s[p];
        bmax = cur.mx[p];
      }
      // FP16 softmax of the lane's four keys
      const half_t mn = hmax(m[p], bmax);
      rr[p] = (float)exp2_h(m[p] - mn);
      prod[p] *= rr[p];
      m[p] = mn;
      const h2_t mn2 = {mn, mn};
      const h2_t p01 = exp2_h2(__builtin_bit_cast(h2_t, s4.x) - mn2);
      const h2_t p23 = exp2_h2(__builtin_bit_cast(h2_t, s4.y) - mn2);
      const float ap[4] = {(float)p01[0], (float)p01[1], (float)p23[0], (float)p23[1]};
      // P^ = HIF4(P) over the row's 64 keys
      const float a4 = fmaxf(fmaxf(ap[0], ap[1]), fmaxf(ap[2], ap[3]));
      const float a8 = fmaxf(a4, __shfl_xor(a4, 1));
      float A = a8;
#pragma unroll
      for (int o = 2; o < 16; o <<= 1) A = fmaxf(A, __shfl_xor(A, o));
      const uint32_t base = e6m2_ceil(A);
      const float bval = e6m2_value(base);
      const bool e2 = a8 <= 0.875f * bval;
      const bool e3 = a4 <= (e2 ? 0.4375f : 0.875f) * bval;
      const int sh = (int)e2 + (int)e3;
      const float R = hif4_rcp_step(base);
      const float C = round_const(sh);
      uint32_t u[4], v[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        u[j] = __float_as_uint(__builtin_fmaf(ap[j], R, C)) - __float_as_uint(C);   // round-half-away(a/step)
        v[j] = u[j] << (2 - sh);
        lp[r * 64 + 16 * quarter + operand_byte(4 * (kq & 3) + j)] = (uint8_t)v[j];
      }
      float ls;
      if (NORM == 0) {
        ls = (float)(v[0] + v[1] + v[2] + v[3]);
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) ls += __shfl_xor(ls, o);
        ls *= bval * 0.0625f;                             // P^ = (4 u 2^-sh) * b/16
      } else {
        ls = (ap[0] + ap[1]) + (ap[2] + ap[3]);
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) ls += __shfl_xor(ls, o);
      }
      l[p] = l[p] * rr[p] + ls;
      sp16[p] = bval * 0.0625f;
      if (DEBUG) {
        const uint64_t b2 = __ballot(e2), b3 = __ballot(e3);
        if (r < grp) {
          const size_t dj = ((size_t)(hk * grp + r) * a.batch + b) * a.NB + J;
          *reinterpret_cast<uint16_t*>(a.dbg_codes + dj * 32 + 2 * kq) =
              (uint16_t)(u[0] | u[1] << 4 | u[2] << 8 | u[3] << 12);
          if (kq == 0) {
            const int l0 = lane & 48;
            uint32_t w2 = 0, w3 = 0;
            for (int k = 0; k < 8; ++k) w2 |= (uint32_t)((b2 >> (l0 + 2 * k)) & 1u) << k;
            for (int k = 0; k < 16; ++k) w3 |= (uint32_t)((b3 >> (l0 + k)) & 1u) << k;
            a.dbg_meta[dj] = base | (w2 << 8) | (w3 << 16);
          }
        }
      }
    }
    // A operands of row n, and the per-row factors of the output rows 4h + c
    i4_t pa0 = {0, 0, 0, 0}, pa1 = {0, 0, 0, 0};
    if (n < grp) {
      pa0 = *reinterpret_cast<const i4_t*>(lp + n * 64 + 32 * h);
      pa1 = *reinterpret_cast<const i4_t*>(lp + n * 64 + 32 * h + 16);
    }
    float rrc[4], spc[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      rrc[c] = __shfl(rr[0], 16 * c);
      spc[c] = __shfl(sp16[0], 16 * c);
      if (RP > 1) {
        const float r1 = __shfl(rr[RP - 1], 16 * c), s1 = __shfl(sp16[RP - 1], 16 * c);
        if (h) {
          rrc[c] = r1;
          spc[c] = s1;
        }
      }
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const uint32_t meta = cur.meta[t];
      const i16_t dot = group_dot(pa0, pa1, cur.w[t], meta, h);
      const float sv = e6m2_value(meta & 255u) * 0.0625f;
#pragma unroll
      for (int c = 0; c < 4; ++c) O[t][c] = __builtin_fmaf(O[t][c], rrc[c], (float)dot[c] * sv * spc[c]);
    }
  };
#pragma unroll
  for (int i = 0; i < kBlocksPerSplit; i += 2) {
    if (J0 + i < J1) block(b0, J0 + i);
    if (i + 2 < kBlocksPerSplit) load(min(J0 + i + 2, J1 - 1), b0);
    if (i + 1 < kBlocksPerSplit && J0 + i + 1 < J1) block(b1, J0 + i + 1);
    if (i + 3 < kBlocksPerSplit) load(min(J0 + i + 3, J1 - 1), b1);
  }
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int r = 4 * h + c;
    if (r < grp) {
      float* dst = a.opart + ((row0 + r) * a.n_split + sp) * D + n;
#pragma unroll
      for (int t = 0; t < NT; ++t) dst[32 * t] = O[t][c];
    }
  }
#pragma unroll
  for (int p = 0; p < RP; ++p) {
    const int r = 4 * p + (lane >> 4);
    if (r < grp && kq == 0)
      a.spart[(row0 + r) * a.n_split + sp] =
          make_float4(lost[p] ? __builtin_nanf("") : l[p], prod[p], (float)m[p], 0.0f);
  }
}

template <int NT, int RP, int NORM, bool DEBUG, int BPS>
__global__ void __launch_bounds__(64 * kMaxWaves, (NT * RP <= 4 ? 4 : 2)) k_decode_split(DecodeArgs a) {
  __shared__ __align__(16) uint8_t lds_p[kMaxWaves][8 * 64];
  WaveSpan w;
  if (!wave_span(a, BPS, w)) return;
  split_run<NT, RP, NORM, DEBUG, BPS, false>(a, w, lds_p[threadIdx.x >> 6], nullptr, nullptr);
}

// ---------------------------------------------------------------------------
// 1+2. Scores and splits in one kernel, once the splits alone fill the chip
// (runs of the split length).  A wave computes its run's scores
// into LDS, publishes each row's maximum over the run (tagged with the call's
// epoch), takes the running maximum entering the run as the maximum of the
// earlier runs' maxima of its sequence, and runs the split from LDS: the
// scores never leave the compute unit.  The earlier runs belong to
// workgroups with lower indices, which each XCD dispatches first, so the
// lowest unfinished workgroup is always running; a spin limit still ends
// every wait.
template <int G, int RP, int NORM, bool DEBUG, int RUN>
__global__ void __launch_bounds__(64 * kMaxWaves, (G * RP <= 2 ? 4 : 2)) k_decode_fused(DecodeArgs a) {
  __shared__ __align__(16) ScoreLds<G, RUN> sl;
  __shared__ __align__(16) uint8_t lds_p[kMaxWaves][8 * 64];
  WaveSpan w;
  if (!wave_span(a, RUN, w)) return;
  const int wave = (int)(threadIdx.x >> 6), lane = threadIdx.x & 63;
  score_run<G, RUN>(a, w, sl);
  const int nb = w.J1 - w.J0;
  if (lane < w.grp && a.publish) {
    half_t rm = sl.m[wave][lane][0];
    for (int i = 1; i < nb; ++i) rm = hmax(rm, sl.m[wave][lane][i]);
    const uint64_t word = ((uint64_t)a.epoch << 32) | (uint64_t)__builtin_bit_cast(uint16_t, rm);
    __hip_atomic_store(a.runmax + (w.row0 + lane) * a.n_split + w.part, word, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  }
  split_run<2 * G, RP, NORM, DEBUG, RUN, true>(a, w, lds_p[wave], &sl.s[wave][0][0], &sl.m[wave][0][0]);
}

// ---------------------------------------------------------------------------
// 3. Merge.  One workgroup per row (b, query head), or per (row, channel
// slice) when there are few rows.  Each split wrote its l,
// the product of its blocks' rescale factors r_J = E(fp16(m_{J-1} - m_J))
// (in block order) and its running maximum after its last block.  Wave 0
// turns the products into R_s = the product over all later splits (a backward
// scan, 64 splits at a time, which also sums l_s R_s); the partial sums,
// loaded before the scan, are then weighted and added, thread (part,
// channel) taking every parts-th split, and the parts combined through LDS.
constexpr int kMergeThreads = 512;

__global__ void __launch_bounds__(kMergeThreads) k_decode_merge(DecodeArgs a) {
  extern __shared__ float R[];                    // [n_split], then partial sums, then the l sum
  const int row = blockIdx.x;                     // b * hq + head
  const int b = row / a.hq, head = row % a.hq;
  const int L = dseq_len(a.cu, b, a.S);
  const int nblk = (L + 63) >> 6;
  if (nblk == 0) return;
  const int ns = (nblk + a.bps - 1) / a.bps;
  const int tid = threadIdx.x, lane = tid & 63;
  // fused path: the splits have read this row's run maxima; clearing them here
  // (a kernel write, so it is part of a captured graph too) means that no word
  // of a finished call can satisfy a later call's wait, whatever its epoch
  if (a.runmax != nullptr && blockIdx.y == 0)
    for (int s = tid; s < ns; s += kMergeThreads) a.runmax[(size_t)row * a.n_split + s] = 0;
  const int D = a.D;
  const int CW = D / (int)gridDim.y;              // this workgroup's channels
  const int parts = kMergeThreads / CW;           // threads per channel
  float* acc_s = R + a.n_split;                   // [parts][CW]
  float* lsum_s = acc_s + parts * CW;
  const float4* sp = a.spart + (size_t)row * a.n_split;
  // the partial sums do not depend on the scan: load them first
  const int c = tid % CW, part = tid / CW, ch = (int)blockIdx.y * CW + c;
  constexpr int kMaxHeld = 16;
  float po[kMaxHeld];
  const float* op = a.opart + (size_t)row * a.n_split * D + ch;
#pragma unroll
  for (int k = 0; k < kMaxHeld; ++k) {
    const int s = part + k * parts;
    po[k] = s < ns ? op[(size_t)s * D] : 0.0f;
  }
  // wave 0: R_s backwards, 64 splits at a time, and l = sum_s l_s R_s
  if (tid < 64) {
    float tail = 1.0f, lpart = 0.0f;
    for (int s1 = ns; s1 > 0; s1 -= 64) {
      const int sidx = s1 - 1 - lane;
      const float4 v = sidx >= 0 ? sp[sidx] : make_float4(0.0f, 1.0f, 0.0f, 0.0f);
      float incl = v.y;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const float t = __shfl_up(incl, o);
        if (lane >= o) incl *= t;
      }
      const float excl = __shfl_up(incl, 1);
      const float rs = tail * (lane == 0 ? 1.0f : excl);
      if (sidx >= 0) {
        R[sidx] = rs;
        lpart = __builtin_fmaf(v.x, rs, lpart);
      }
      tail *= __shfl(incl, 63);
    }
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) lpart += __shfl_xor(lpart, o);
    if (lane == 0) lsum_s[0] = lpart;
  }
  __syncthreads();
  float acc = 0.0f;
#pragma unroll
  for (int k = 0; k < kMaxHeld; ++k) {
    const int s = part + k * parts;
    if (s < ns) acc = __builtin_fmaf(po[k], R[s], acc);
  }
  for (int s = part + kMaxHeld * parts; s < ns; s += parts) acc = __builtin_fmaf(op[(size_t)s * D], R[s], acc);
  acc_s[part * CW + c] = acc;
  __syncthreads();
  if (part == 0) {
    float o = acc;
    for (int p = 1; p < parts; ++p) o += acc_s[p * CW + c];
    const float lsum = lsum_s[0];
    a.o[(size_t)row * D + ch] = (half_t)(o * (1.0f / lsum));
    if (ch == 0) a.lse[(size_t)head * a.batch + b] = sp[ns - 1].z * 0.69314718055994531f + logf(lsum);
  }
}

int pick_run(int head_groups, int batch, int NB) {
  for (int run : kScoreRuns)
    if ((long)head_groups * batch * ((NB + run - 1) / run) >= kMinScoreWorkgroups) return run;
  return 1;
}

int pick_split(int head_groups, int batch, int NB) {
  int pick = kSplitLengths[0];
  for (int bps : kSplitLengths) {
    const int n_split = (NB + bps - 1) / bps;
    if (bps != kSplitLengths[0] && n_split > kMaxSplitsPerRow) break;
    pick = bps;
    if ((long)head_groups * batch * n_split >= kMinSplitWorkgroups) break;
  }
  return pick;
}

int maxima_stride(int NB) { return (NB + 7) & ~7; }

struct DecodePlan {
  int waves, head_groups, run, bps;
  bool fused;              // one kernel for scores and splits
};

DecodePlan plan_decode(int batch, int hkv, int NB) {
  DecodePlan p;
  p.waves = hkv < kMaxWaves ? hkv : kMaxWaves;
  p.head_groups = (hkv + p.waves - 1) / p.waves;
  p.run = pick_run(p.head_groups, batch, NB);
  p.bps = pick_split(p.head_groups, batch, NB);
  // one kernel for scores and splits once the splits fill the chip; below
  // that the score kernel's shorter runs give the score phase more workgroups
  p.fused = (long)p.head_groups * batch * ((NB + p.bps - 1) / p.bps) >= kMinSplitWorkgroups;
  return p;
}

void decode_offsets(int batch, int hq, int D, int NB, const DecodePlan& pl, size_t off[6]) {
  const size_t rows = (size_t)batch * hq;
  const int n_split = (NB + pl.bps - 1) / pl.bps;
  size_t o = 0;
  off[0] = o; o += pl.fused ? 0 : round_up256(rows * NB * 64 * 2);             // scores
  off[1] = o; o += pl.fused ? 0 : round_up256(rows * maxima_stride(NB) * 2);   // block maxima
  off[2] = o; o += round_up256(rows * n_split * D * 4);                         // partial O
  off[3] = o; o += round_up256(rows * n_split * 16);                            // l, factor product, max
  off[4] = o; o += pl.fused ? round_up256(rows * n_split * 8) : 0;              // run maxima
  off[5] = o;
}

// Epoch tags of the fused path: a fresh value per call, starting from a
// random point.  Tags only separate eager calls; under graph replay the tag
// is the captured one, and what keeps a replay from reading the previous
// replay's words is the merge kernel clearing them (a cleared word never
// matches, the tag is never 0).
uint32_t next_epoch() {
  static std::atomic<uint32_t> counter{(uint32_t)std::random_device{}()};
  uint32_t e = counter.fetch_add(1) + 1;
  if (e == 0) e = counter.fetch_add(1) + 1;
  return e;
}

template <typename K>
hipError_t allow_lds(K kern, size_t bytes) {
  if (bytes <= 65536) return hipSuccess;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)bytes);
}

template <int NT, int RP, int BPS>
void launch_split(const DecodeArgs& a, int norm, bool debug, dim3 grid, dim3 block, hipStream_t st) {
  if (norm == 0) {
    if (debug) k_decode_split<NT, RP, 0, true, BPS><<<grid, block, 0, st>>>(a);
    else k_decode_split<NT, RP, 0, false, BPS><<<grid, block, 0, st>>>(a);
  } else {
    if (debug) k_decode_split<NT, RP, 1, true, BPS><<<grid, block, 0, st>>>(a);
    else k_decode_split<NT, RP, 1, false, BPS><<<grid, block, 0, st>>>(a);
  }
}

template <int NT, int BPS>
void launch_split_rows(const DecodeArgs& a, int grp, int norm, bool debug, dim3 grid, dim3 block,
                       hipStream_t st) {
  if (grp <= 4) launch_split<NT, 1, BPS>(a, norm, debug, grid, block, st);
  else launch_split<NT, 2, BPS>(a, norm, debug, grid, block, st);
}

template <int NT>
void launch_split_run(const DecodeArgs& a, int grp, int norm, bool debug, dim3 grid, dim3 block,
                      hipStream_t st) {
  switch (a.bps) {
    case 8: launch_split_rows<NT, 8>(a, grp, norm, debug, grid, block, st); break;
    case 4: launch_split_rows<NT, 4>(a, grp, norm, debug, grid, block, st); break;
    default: launch_split_rows<NT, 2>(a, grp, norm, debug, grid, block, st); break;
  }
}

template <int G, int RP, int RUN>
void launch_fused_run(const DecodeArgs& a, int norm, bool debug, dim3 grid, dim3 block, hipStream_t st) {
  if (norm == 0) {
    if (debug) k_decode_fused<G, RP, 0, true, RUN><<<grid, block, 0, st>>>(a);
    else k_decode_fused<G, RP, 0, false, RUN><<<grid, block, 0, st>>>(a);
  } else {
    if (debug) k_decode_fused<G, RP, 1, true, RUN><<<grid, block, 0, st>>>(a);
    else k_decode_fused<G, RP, 1, false, RUN><<<grid, block, 0, st>>>(a);
  }
}

template <int G, int RP>
void launch_fused_rows(const DecodeArgs& a, int norm, bool debug, dim3 grid, dim3 block, hipStream_t st) {
  switch (a.bps) {
    case 8: launch_fused_run<G, RP, 8>(a, norm, debug, grid, block, st); break;
    case 4: launch_fused_run<G, RP, 4>(a, norm, debug, grid, block, st); break;
    default: launch_fused_run<G, RP, 2>(a, norm, debug, grid, block, st); break;
  }
}

template <int G>
void launch_fused(const DecodeArgs& a, int grp, int norm, bool debug, dim3 grid, dim3 block, hipStream_t st) {
  if (grp <= 4) launch_fused_rows<G, 1>(a, norm, debug, grid, block, st);
  else launch_fused_rows<G, 2>(a, norm, debug, grid, block, st);
}

template <int G>
void launch_scores(const DecodeArgs& a, int run, dim3 block, hipStream_t st) {
  const int head_groups = (a.hkv + a.waves - 1) / a.waves;
  const dim3 grid(head_groups, (a.NB + run - 1) / run, a.batch);
  switch (run) {
    case 8: k_decode_scores<G, 8><<<grid, block, 0, st>>>(a); break;
    case 2: k_decode_scores<G, 2><<<grid, block, 0, st>>>(a); break;
    default: k_decode_scores<G, 1><<<grid, block, 0, st>>>(a); break;
  }
}

}  // namespace

size_t decode_workspace_bytes(int batch, int hq, int hkv, int D, int NB) {
  size_t off[6];
  decode_offsets(batch, hq, D, NB, plan_decode(batch, hkv, NB), off);
  return off[5];
}

hipError_t launch_decode(const DecodeLaunch& d, hipStream_t st) {
  const DecodePlan pl = plan_decode(d.batch, d.hkv, d.NB);
  const int waves = pl.waves, head_groups = pl.head_groups, run = pl.run, bps = pl.bps;
  size_t off[6];
  decode_offsets(d.batch, d.hq, d.D, d.NB, pl, off);
  uint8_t* ws = d.ws;
  DecodeArgs a;
  a.q = d.q;
  a.s = d.s;
  a.kc = d.kc;
  a.km = d.km;
  a.vc = d.vc;
  a.vm = d.vm;
  a.cu = d.cu;
  a.s2 = reinterpret_cast<half_t*>(ws + off[0]);
  a.mx = reinterpret_cast<half_t*>(ws + off[1]);
  a.opart = reinterpret_cast<float*>(ws + off[2]);
  a.spart = reinterpret_cast<float4*>(ws + off[3]);
  a.runmax = pl.fused ? reinterpret_cast<uint64_t*>(ws + off[4]) : nullptr;
  a.epoch = pl.fused ? next_epoch() : 0;
  a.spin_limit = d.test_no_publish ? 16 : kSpinLimit;
  a.publish = d.test_no_publish ? 0 : 1;
  a.o = d.o;
  a.lse = d.lse;
  a.dbg_codes = d.dbg_codes;
  a.dbg_meta = d.dbg_meta;
  a.batch = d.batch;
  a.S = d.S;
  a.NB = d.NB;
  a.hq = d.hq;
  a.hkv = d.hkv;
  a.D = d.D;
  a.bps = bps;
  a.n_split = (d.NB + bps - 1) / bps;
  a.mxs = maxima_stride(d.NB);
  a.waves = waves;
  a.c = d.c;
  const int grp = d.hq / d.hkv;
  hipError_t e;
  const dim3 block(64 * a.waves);
  const dim3 g2(head_groups, a.n_split, d.batch);
  const bool dbg = d.dbg_codes != nullptr;
  if (pl.fused) {
    switch (d.D) {
      case 64: launch_fused<1>(a, grp, d.norm, dbg, g2, block, st); break;
      case 128: launch_fused<2>(a, grp, d.norm, dbg, g2, block, st); break;
      default: launch_fused<4>(a, grp, d.norm, dbg, g2, block, st); break;
    }
  } else {
    switch (d.D) {
      case 64: launch_scores<1>(a, run, block, st); break;
      case 128: launch_scores<2>(a, run, block, st); break;
      default: launch_scores<4>(a, run, block, st); break;
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    switch (d.D) {
      case 64: launch_split_run<2>(a, grp, d.norm, dbg, g2, block, st); break;
      case 128: launch_split_run<4>(a, grp, d.norm, dbg, g2, block, st); break;
      default: launch_split_run<8>(a, grp, d.norm, dbg, g2, block, st); break;
    }
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (d.ev && (e = hipEventRecord(d.ev[1], st)) != hipSuccess) return e;
  // few rows: each row's channels are split over several workgroups (at
  // least 32 channels each), so that every thread holds few partials
  const long rows = (long)d.batch * d.hq;
  int slices = 1;
  while (rows * slices < kMinSplitWorkgroups && d.D / (2 * slices) >= 32) slices *= 2;
  const size_t lds3 = ((size_t)a.n_split + kMergeThreads + 1) * sizeof(float);
  if ((e = allow_lds(k_decode_merge, lds3)) != hipSuccess) return e;
  k_decode_merge<<<dim3((unsigned)rows, slices), dim3(kMergeThreads), lds3, st>>>(a);
  return hipGetLastError();
}

}  // namespace hifa4
