// Internal declarations shared by the HIP translation units of libhifa4.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace hifa4 {

typedef _Float16 half_t;

// Byte layout of one pre-pass chunk = (sequence, kv head, 64-key block).
// Offsets are multiples of 256 bytes.
// An FP6 MFMA operand of one wave (64 lanes x 24 bytes) as stored in a chunk:
// the first 16 bytes of every lane, then the last 8 bytes of every lane.
constexpr size_t kOpRecord = 64 * 24;

struct ChunkLayout {
  size_t k_op, k_scale, v_op, v_scale, kappa, bytes;
};

__host__ __device__ constexpr size_t round_up256(size_t x) { return (x + 255) & ~(size_t)255; }

// HIF4 operands, each group as the two MFMA operands of its split base
// (operand A = codes, B = zero, codes or negated codes; byte 0 / 1 of the
// scale word are their E8M0 scales):
//   K [2 halves][G][2 operands] records, K scale words [2][G][32 keys],
//   V [D/32][2 operands] records, V scale words [D],
//   with Q-Mean: kappa [64 keys] fp32, the exact channel sum of each smoothed
//   key rounded once.
__host__ __device__ constexpr ChunkLayout chunk_layout_hif4(int G, bool qmean = false) {
  ChunkLayout c{};
  c.k_op = 0;
  c.k_scale = round_up256((size_t)2 * G * 2 * kOpRecord);
  c.v_op = c.k_scale + round_up256((size_t)2 * G * 32 * 4);
  c.v_scale = c.v_op + round_up256((size_t)(2 * G) * 2 * kOpRecord);
  c.kappa = c.v_scale + round_up256((size_t)64 * G * 4);
  const size_t end = c.kappa + (qmean ? round_up256((size_t)64 * 4) : 0);
  // a multiple of 1 KiB: the attention kernel streams chunks into LDS in
  // whole-wave pieces of 64 lanes x 16 bytes
  c.bytes = (end + 1023) & ~(size_t)1023;
  return c;
}

// FP16 operands: K [2][D/16][64][16 B], V [D/32][4][64][16 B].
__host__ __device__ constexpr ChunkLayout chunk_layout_fp16(int D) {
  ChunkLayout c{};
  c.k_op = 0;
  c.k_scale = c.k_op + round_up256((size_t)2 * (D / 16) * 64 * 16);
  c.v_op = c.k_scale;
  c.v_scale = c.v_op + round_up256((size_t)(D / 32) * 4 * 64 * 16);
  c.bytes = c.v_scale;
  return c;
}

struct AttnArgs {
  const half_t* q;
  const float* s;          // smoothing scales or nullptr
  const int* cu;           // cu_seqlens or nullptr
  const uint8_t* ws;       // pre-pass chunks
  half_t* o;
  float* lse;
  uint8_t* dbg_codes;      // optional P^ dump [dbg_nh, dbg_nt, NB, 32]
  uint32_t* dbg_meta;      // [dbg_nh, dbg_nt, NB]
  int dbg_h0, dbg_nh;      // dumped query heads [dbg_h0, dbg_h0 + dbg_nh)
  int dbg_t0, dbg_nt;      // dumped tokens [dbg_t0, dbg_t0 + dbg_nt)
  int batch, S, NB, hq, hkv, D, total_tokens;
  float c;                 // log2(e)/sqrt(D)
};

// Entry of the P^ dump for (query head, token, block), false outside the
// dumped window.
__device__ __forceinline__ bool dbg_entry(const AttnArgs& a, int hq, int tok, int J, size_t& e) {
  const int hr = hq - a.dbg_h0, tr = tok - a.dbg_t0;
  if ((unsigned)hr >= (unsigned)a.dbg_nh || (unsigned)tr >= (unsigned)a.dbg_nt) return false;
  e = ((size_t)hr * a.dbg_nt + tr) * a.NB + J;
  return true;
}

hipError_t launch_quant_rows(const half_t* x, const float* s, uint8_t* codes, uint32_t* meta, long n_rows,
                             int heads, int heads_kv, int D, bool is_k, hipStream_t st);
hipError_t launch_quant_v(const half_t* v, const int* cu, uint8_t* codes, uint32_t* meta, int batch, int S, int NB,
                          int heads_kv, int D, hipStream_t st);
hipError_t launch_prep_kv(const half_t* k, const half_t* v, const float* s, const int* cu, uint8_t* ws, int batch,
                          int S, int NB, int heads_kv, int D, bool fp16, bool qmean, hipStream_t st);
hipError_t launch_calib(const half_t* q, const half_t* k, int n, int S, int hq, int hkv, int D, uint32_t* stats,
                        unsigned long long* hist, hipStream_t st);
hipError_t launch_selftest_exp2(const half_t* x, half_t* y, long n, hipStream_t st);
// operands: 0 HIF4, 1 FP16 reference, 2 P-only (fp16 Q, K, V; HIF4 P)
hipError_t launch_attention(const AttnArgs& a, int norm, int operands, bool qmean, hipStream_t st);

}  // namespace hifa4
