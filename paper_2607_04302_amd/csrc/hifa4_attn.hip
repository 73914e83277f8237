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
//     and 32-key half (the A operands are the pre-pass K records in LDS, whose
//     E8M0 scales carry b_K exactly; B is the Q tile quantized in registers at
//     kernel start); each group sum is exact, the fp32 epilogue forms each
//     group's exact term (times b_Q/4), sums the groups in order in fp32,
//     multiplies by the score scale c in fp32 and rounds to fp16.  In S^T
//     each lane holds one query and 32 of the block's keys, so row maxima are
//     in-lane plus one exchange with lane l^32;
//   FP16 softmax: m_new = max(m, rowmax), P = 2^(S2 - m_new), r = 2^(m - m_new);
//   P^ = HIF4(P) in registers: the lane's 32 keys are 8 complete 4-key blocks,
//     8-key blocks pair with lane l^32; values become FP6 operands directly;
//   O^T[d, q] += V^T P^T: the lane's P^ values already form the B operand of
//     the 32x32x64 MFMA (the pre-pass stored V^ in the matching key order, as
//     two operands per group whose scales carry b_V), an fp32 epilogue
//     applies b_P and the deferred rescale; the normalizer comes out of one
//     more MFMA against an all-ones A operand (the [V^ | 1] column of the
//     paper).
#include "hifa4_device.h"
#include "hifa4_internal.h"
#include "hifa4_packed.h"

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
  m.L = a.cu ? min(a.cu[m.b + 1] - m.t0, a.S) : a.S;     // lengths above max_seqlen are clamped (outside the contract)
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

// A wave-uniform pointer read into scalar registers (its value is the same in
// every lane; the compiler cannot see that for values derived from the wave
// index).
__device__ __forceinline__ const uint8_t* uniform_ptr(const uint8_t* p) {
  const uint64_t u = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
  return reinterpret_cast<const uint8_t*>(((uint64_t)hi << 32) | lo);
}

// Asynchronous copy of one chunk (BYTES, a multiple of 1 KiB) from global
// memory straight into LDS (global_load_lds, 16 bytes per lane; lane i of a
// wave lands at the wave's LDS base + 16 i), in pieces of 256 lanes x 16
// bytes.  On the last block of a tile the current chunk is streamed into the
// idle buffer again, which keeps the block code free of branches.
// Completion is tracked by vmcnt: the caller waits with vmcnt(0) and a
// barrier before reading.  Issuing a piece stalls the wave while the texture
// path is busy, so the block code spreads the pieces over its phases instead
// of issuing the whole chunk at once.  The load is written out (M0 set to the
// wave's LDS destination, the global base in scalar registers, the lane's
// 16-byte offset in one VGPR) because the compiler forms the address of the
// builtin form with 64-bit vector adds per piece; the hardware counts these
// loads in vmcnt like any other and completes them in issue order.  The
// compiler treats M0 as reserved and keeps no value of its own there across
// the statement, so nothing else in this file may use M0
// (tests/test_m0_guard.py checks the compiled code).
struct ChunkStream {
  uint8_t* dst;            // LDS buffer
  const uint8_t* src;      // global chunk (the last block streams a copy of itself)
  int wave;                // wave index in the workgroup (uniform)
};

template <int BYTES>
__device__ __forceinline__ void stream_piece(const ChunkStream& cs, int r) {
  constexpr int n16 = BYTES / 16;
  if (r * 256 >= n16) return;
  // every piece but possibly the last covers all four waves (n16 is a
  // multiple of 64); the conditions are uniform, so no lane masking
  if (256 * (r + 1) > n16 && 256 * r + 64 * cs.wave >= n16) return;
  // global_load_lds_dwordx4 with a scalar base: lane i reads 16 bytes at
  // base + 16 i and writes them to LDS at M0 + 16 i
  const uint8_t* gbase = cs.src + (4096 * r + 1024 * cs.wave);
  uint8_t* const ldst = cs.dst + 4096 * r + 1024 * cs.wave;
  const uint32_t m0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)ldst;
  const uint32_t voff = 16u * (threadIdx.x & 63u);
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(gbase), "s"(m0)
               : "memory", "m0");
}

template <int BYTES>
__device__ __forceinline__ void stream_pieces_from(const ChunkStream& cs, int r0) {
#pragma unroll
  for (int r = r0; r < (BYTES / 16 + 255) / 256; ++r) stream_piece<BYTES>(cs, r);
}

template <int BYTES>
__device__ __forceinline__ void stage_chunk_async(uint8_t* lds, const uint8_t* __restrict__ g) {
  stream_pieces_from<BYTES>(ChunkStream{lds, g, __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6))}, 0);
}

__device__ __forceinline__ void wait_async_copies() { __builtin_amdgcn_s_waitcnt(0x0F70); }   // vmcnt(0)

// vmcnt(N): at most N vector-memory operations of the wave outstanding (they
// complete in issue order).  gfx9 encoding: vmcnt low bits [3:0], high bits
// [15:14]; expcnt and lgkmcnt left at their maxima.
template <int N>
__device__ __forceinline__ void wait_vmcnt_k() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | 0x0F70);
}

// One lane's 24-byte FP6 operand from an operand record (64 lanes x 16
// bytes, then 64 lanes x 8 bytes).  The 8-byte tail is read through a volatile
// access so that the compiler does not pair it with the tail of another
// operand into one 16-byte read, which would cost register copies to rebuild
// the contiguous 6-register MFMA operand.
__device__ __forceinline__ i8_t ld_op6(const uint8_t* rec, int lane) {
  typedef uint32_t u2_t __attribute__((ext_vector_type(2)));
  typedef uint32_t u4v_t __attribute__((ext_vector_type(4)));
  typedef const volatile __attribute__((address_space(3))) u2_t lds_u2_t;
  const u4v_t a = *reinterpret_cast<const u4v_t*>(rec + 16 * lane);
  const u2_t c = *(lds_u2_t*)(rec + 1024 + 8 * lane);
  i8_t r;
  r[0] = (int)a.x; r[1] = (int)a.y; r[2] = (int)a.z; r[3] = (int)a.w; r[4] = (int)c.x; r[5] = (int)c.y;
  r[6] = 0; r[7] = 0;
  return r;
}

__device__ __forceinline__ f16v_t mfma6(const i8_t& A, const i8_t& B, const f16v_t& C) {
  // FP6 E2M3 x FP6 E2M3, unit E8M0 scales (127 = 2^0).
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(A, B, C, 2, 2, 0, 127, 0, 127);
}

__device__ __forceinline__ half_t hmax(half_t a, half_t b) { return a > b ? a : b; }

// FP6 x FP6 MFMA whose A rows are scaled by byte OPSEL of `sa` (B unscaled).
template <int OPSEL>
__device__ __forceinline__ f16v_t mfma6_rows(const i8_t& A, const i8_t& B, const f16v_t& C, int sa) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(A, B, C, 2, 2, OPSEL, sa, 0, 127);
}

// Global key index (within the 64-key block) held by lane half h at tile t,
// accumulator register v of the 32x32 output layout.
__device__ __forceinline__ int key_of(int t, int h, int v) { return 32 * t + 8 * (v >> 2) + 4 * h + (v & 3); }

// ---------------------------------------------------------------------------
// HiFA4 kernel.
//
// K/V chunks alternate between two LDS buffers: while block J is consumed,
// chunk J+1 streams into the other buffer (global_load_lds), and the block's
// closing barrier waits for it.  At D=128 three waves per SIMD (three
// workgroups per CU) let one wave's MFMAs and memory waits run under the
// others' vector work.  The block that holds a wave's diagonal is processed by
// a separate instantiation (MASK) so that the causal mask costs nothing on the
// other blocks.
//
// Scores: for each 32-key half t and channel group g two MFMAs accumulate
// K^'s codes and the second operand of the split base (zero, the codes or the
// negated codes), with E8M0 row scales that together make K's exact b/4; the
// result is the exact sum of o_q * (o_k * b_k/4) in fp32.  V^ enters the PV
// product the same way, so its groups are exact too.  The epilogue
// multiplies by the lane's own b_q/4 (each lane owns one query in S^T), which
// gives the group's exact term t_g; the terms are summed in order in fp32 (a
// fused multiply-add of the exact product rounds exactly the sum), the sum
// is multiplied by c, then rounded to fp16: G + 1 VALU operations per score
// plus the fp16 rounding.
//
// Deferred rescale: instead of O <- r*O every block, the kernel keeps
// O* = O / rho and l* = l / rho with rho the product of the rescale factors so
// far, and adds each block's contribution scaled by 1/rho.  O*/l* = O/l, so
// the output and the P^ codes are unchanged; only the fp32 rounding of O
// differs.  A factor r = 0 (a running max that grows by more than 24 in log2
// units after the first block) wipes the history, exactly as r*O does.

// Wave issue priority from the work left.  A SIMD issues from the oldest
// ready wave first, so without this the youngest of the co-resident
// workgroups (the one dispatched last) is starved and finishes last even
// when it has the least work.  Raising the priority of the workgroups with
// the most blocks left makes the co-resident workgroups of a CU finish
// together (longest remaining work first).
__device__ __forceinline__ void set_priority_by_work_left(int blocks_left) {
  const int p = blocks_left >= 48 ? 3 : (blocks_left >= 24 ? 2 : (blocks_left >= 8 ? 1 : 0));
  switch (p) {
    case 3: __builtin_amdgcn_s_setprio(3); break;
    case 2: __builtin_amdgcn_s_setprio(2); break;
    case 1: __builtin_amdgcn_s_setprio(1); break;
    default: __builtin_amdgcn_s_setprio(0); break;
  }
}

// fp16 exponential of four packed pairs; the four low-half results are
// written before the first SDWA high-half instruction reads its destination,
// which keeps the transcendental result latency out of the way without nops.
__device__ __forceinline__ void exp2_h2x4(const h2_t x[4], h2_t y[4]) {
  asm("v_exp_f16 %0, %4\n\t"
      "v_exp_f16 %1, %5\n\t"
      "v_exp_f16 %2, %6\n\t"
      "v_exp_f16 %3, %7\n\t"
      "v_exp_f16_sdwa %0, %4 dst_sel:WORD_1 dst_unused:UNUSED_PRESERVE src0_sel:WORD_1\n\t"
      "v_exp_f16_sdwa %1, %5 dst_sel:WORD_1 dst_unused:UNUSED_PRESERVE src0_sel:WORD_1\n\t"
      "v_exp_f16_sdwa %2, %6 dst_sel:WORD_1 dst_unused:UNUSED_PRESERVE src0_sel:WORD_1\n\t"
      "v_exp_f16_sdwa %3, %7 dst_sel:WORD_1 dst_unused:UNUSED_PRESERVE src0_sel:WORD_1"
      : "=&v"(y[0]), "=&v"(y[1]), "=&v"(y[2]), "=&v"(y[3])
      : "v"(x[0]), "v"(x[1]), "v"(x[2]), "v"(x[3]));
}

// Packed maximum of 16 pairs (a tree of 15 v_pk_max_f16 in one block).
__device__ __forceinline__ h2_t hmax16(const h2_t x[16]) {
  h2_t y, a1, a2, a3, a4, a5, a6, a7;
  asm("v_pk_max_f16 %0, %8, %9\n\t"
      "v_pk_max_f16 %1, %10, %11\n\t"
      "v_pk_max_f16 %2, %12, %13\n\t"
      "v_pk_max_f16 %3, %14, %15\n\t"
      "v_pk_max_f16 %4, %16, %17\n\t"
      "v_pk_max_f16 %5, %18, %19\n\t"
      "v_pk_max_f16 %6, %20, %21\n\t"
      "v_pk_max_f16 %7, %22, %23\n\t"
      "v_pk_max_f16 %0, %0, %1\n\t"
      "v_pk_max_f16 %2, %2, %3\n\t"
      "v_pk_max_f16 %4, %4, %5\n\t"
      "v_pk_max_f16 %6, %6, %7\n\t"
      "v_pk_max_f16 %0, %0, %2\n\t"
      "v_pk_max_f16 %4, %4, %6\n\t"
      "v_pk_max_f16 %0, %0, %4"
      : "=&v"(y), "=&v"(a1), "=&v"(a2), "=&v"(a3), "=&v"(a4), "=&v"(a5), "=&v"(a6), "=&v"(a7)
      : "v"(x[0]), "v"(x[1]), "v"(x[2]), "v"(x[3]), "v"(x[4]), "v"(x[5]), "v"(x[6]), "v"(x[7]), "v"(x[8]),
        "v"(x[9]), "v"(x[10]), "v"(x[11]), "v"(x[12]), "v"(x[13]), "v"(x[14]), "v"(x[15]));
  return y;
}
// Raw inputs of one query half-group: the lane's 32 fp16 values and, with
// Smooth-QK, its 32 scales.
struct QRaw {
  h2_t x[16];
  float4 s[8];
};

__device__ __forceinline__ void load_q_half_group(const half_t* __restrict__ src, const float* __restrict__ sp,
                                                  bool row_ok, QRaw& r) {
  typedef uint32_t u4v_t __attribute__((ext_vector_type(4)));
  if (row_ok) {
    const u4v_t* p = reinterpret_cast<const u4v_t*>(src);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const u4v_t w = p[v];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        // copy the element first: bit-casting an ext_vector element in place
        // makes clang read element 0 for every i
        const uint32_t wi = w[i];
        r.x[4 * v + i] = __builtin_bit_cast(h2_t, wi);
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) r.x[i] = h2_t{(half_t)0, (half_t)0};
  }
  if (sp) {
    const float4* s4 = reinterpret_cast<const float4*>(sp);
#pragma unroll
    for (int v = 0; v < 8; ++v) r.s[v] = s4[v];
  } else {
    // defined on every path, so that no undefined value is carried anywhere
#pragma unroll
    for (int v = 0; v < 8; ++v) r.s[v] = make_float4(1.0f, 1.0f, 1.0f, 1.0f);
  }
}

// Smooth-QK of the raw half-group: fp16(q*s) per element (or q unchanged).
__device__ __forceinline__ void smooth_half_group(const QRaw& r, bool smooth, h2_t x[16]) {
#pragma unroll
  for (int i = 0; i < 16; ++i) x[i] = r.x[i];
  if (smooth) {
#pragma unroll
    for (int v = 0; v < 8; ++v) {
      x[2 * v] = smooth_mul2(x[2 * v], r.s[v].x, r.s[v].y);
      x[2 * v + 1] = smooth_mul2(x[2 * v + 1], r.s[v].z, r.s[v].w);
    }
  }
}

// Q-Mean (Algorithm 1, the mean step): mu = fp16(sum of the row's D smoothed
// values / D), the sum exact in float64, then Q_z = fp16(q~ - mu) in place
// (one packed fp16 subtraction per pair, each difference rounded once).
// The lane pair (l, l^32) holds the row; returns mu as fp32 (exact).
template <int G>
__device__ __forceinline__ float centre_q_row(h2_t (&x)[G][16]) {
  double part = 0.0;
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int i = 0; i < 16; ++i) part += (double)(float)x[g][i][0] + (double)(float)x[g][i][1];
  part += __shfl_xor(part, 32);
  const half_t mu = rn16_from_f64(part * (1.0 / (64.0 * G)));
  const h2_t mu2 = {mu, mu};
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int i = 0; i < 16; ++i) x[g][i] = x[g][i] - mu2;
  return (float)mu;
}

// HIF4 of one query group (row layout, see rows_quantize): the lane's FP6 B
// operand and the group's scale b/4 (exact), which turns the MFMA's group
// dot into the group's exact score term.
__device__ __forceinline__ void quantize_q_half_group(const h2_t (&x)[16], i8_t& qop, float& wq) {
  const GroupOps r = rows_quantize(x);
#pragma unroll
  for (int i = 0; i < 6; ++i) qop[i] = r.pk[i];
  qop[6] = 0;
  qop[7] = 0;
  wq = 0.25f * r.bval;
}

template <int G>
struct Hif4State {
  f16v_t O[2 * G];
  half_t m_run;
  float l_star;     // l / rho (consistent or mismatched per NORM)
  float inv_rho;    // 1 / rho
};

template <int G, int NORM, bool DEBUG, bool QMEAN, bool MASK>
__device__ __forceinline__ void hif4_block(const AttnArgs& a, const TileMap& tm, const uint8_t* cur, int J, int lane,
                                           int h, int col, int qi, bool row_ok, const i8_t (&qop)[G],
                                           const float (&wq)[G], float cmu, const i8_t& ones, Hif4State<G>& st,
                                           const ChunkStream& cs) {
  constexpr int DT = 2 * G;
  constexpr ChunkLayout lay = chunk_layout_hif4(G, QMEAN);
  constexpr int CB = (int)lay.bytes;
  // ---- scores: S2 = fp16(fp32(S_acc * c)), S_acc the fp32 sum of the exact
  // group terms t_g = d_g * b_q,g/4 in group order (with Q-Mean, then
  // fp32(S_acc + mu kappa_j)); a fused multiply-add of an exact product
  // rounds exactly the sum.
  h2_t s2[2][8];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    stream_piece<CB>(cs, t);
    f16v_t acc[G];
    int ks[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      ks[g] = reinterpret_cast<const int*>(cur + lay.k_scale)[(t * G + g) * 32 + col];
      const f16v_t c0 = {};
      acc[g] = mfma6_rows<0>(ld_op6(cur + lay.k_op + (size_t)((t * G + g) * 2 + 0) * kOpRecord, lane), qop[g], c0,
                             ks[g]);
    }
#pragma unroll
    for (int g = 0; g < G; ++g)
      acc[g] = mfma6_rows<1>(ld_op6(cur + lay.k_op + (size_t)((t * G + g) * 2 + 1) * kOpRecord, lane), qop[g],
                             acc[g], ks[g]);
    stream_piece<CB>(cs, 2 + t);
    float sacc[16];
    if (QMEAN) {
      // the Q-Mean correction mu * kappa_j of the lane's keys 32t + 8j + 4h +
      // [0, 4) follows the group terms, four keys at a time so that the key
      // sums occupy no more registers than the dying accumulators
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float4 kp = *reinterpret_cast<const float4*>(cur + lay.kappa + 4 * (32 * t + 8 * j + 4 * h));
        const float kv[4] = {kp.x, kp.y, kp.z, kp.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float x = acc[0][4 * j + i] * wq[0];
#pragma unroll
          for (int g = 1; g < G; ++g) x = __builtin_fmaf(acc[g][4 * j + i], wq[g], x);
          x = __builtin_fmaf(cmu, kv[i], x);
          sacc[4 * j + i] = x * a.c;
        }
      }
    } else {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float x = acc[0][v] * wq[0];
#pragma unroll
        for (int g = 1; g < G; ++g) x = __builtin_fmaf(acc[g][v], wq[g], x);
        sacc[v] = x * a.c;
      }
    }
#pragma unroll
    for (int v2 = 0; v2 < 8; ++v2) s2[t][v2] = pack2_f16(sacc[2 * v2], sacc[2 * v2 + 1]);
  }
  if (MASK) {
    const half_t ninf = (half_t)(-__builtin_inff());
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        if (64 * J + key_of(t, h, v) > qi) s2[t][v >> 1][v & 1] = ninf;
  }
  // ---- running max (FP16), exchanged with lane l^32.
  h2_t mx2 = hmax16(&s2[0][0]);
  mx2 = hmax_halves(max_with_partner(mx2));            // block row max, both halves
  const h2_t mr2 = {st.m_run, st.m_run};
  const h2_t mn2 = hmax2(mr2, mx2);                    // m_new, both halves
  stream_piece<CB>(cs, 4);
  // ---- P = 2^(S2 - m_new); r = 2^(m - m_new) and the block max A = 2^(mx - m_new).
  h2_t p2[2][8];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      h2_t xin[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) xin[i] = s2[t][4 * q + i] - mn2;
      exp2_h2x4(xin, &p2[t][4 * q]);
    }
  const h2_t ra = exp2_h2(h2_t{mr2[0], mx2[0]} - mn2);
  const float r = (float)ra[0];
  const float A = (float)ra[1];
  st.m_run = mn2[0];

  float psum = 0.0f;
  if (NORM == 1) {
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int v2 = 0; v2 < 8; ++v2) psum = __builtin_amdgcn_fdot2(p2[t][v2], h2_t{(half_t)1, (half_t)1}, psum, false);
    psum = add_with_partner(psum);
  }

  stream_piece<CB>(cs, 5);
  // ---- P^ = HIF4(P) over the block's 64 keys (P-Reordering).
  uint8_t* dcodes = nullptr;
  uint32_t* dmeta = nullptr;
  size_t e;
  if (DEBUG && row_ok && dbg_entry(a, tm.hq, tm.t0 + qi, J, e)) {
    dcodes = a.dbg_codes + e * 32;
    dmeta = a.dbg_meta + e;
  }
  const PQuant pq = quantize_p_block<DEBUG>(p2, A, lane, h, dcodes, dmeta);
  const float bval = pq.bval;
  const i6_t pk = __builtin_amdgcn_cvt_scalef32_pk32_fp6_f16(pq.ov, 1.0f);
  i8_t pop;
#pragma unroll
  for (int i = 0; i < 6; ++i) pop[i] = pk[i];
  pop[6] = 0;
  pop[7] = 0;

  stream_piece<CB>(cs, 6);
  // ---- deferred rescale bookkeeping (lane-uniform factors).
  if (__builtin_expect(J > 0 && __builtin_amdgcn_ballot_w64(r == 0.0f) != 0, 0)) {
    // history wiped for some rows: O <- 0*O, l <- 0*l there
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int v = 0; v < 16; ++v) st.O[dt][v] = r == 0.0f ? 0.0f : st.O[dt][v];
    st.l_star = r == 0.0f ? 0.0f : st.l_star;
  }
  st.inv_rho = (r == 0.0f) ? 1.0f : st.inv_rho * __builtin_amdgcn_rcpf(r);
  if (__builtin_expect(__builtin_amdgcn_ballot_w64(st.inv_rho > 0x1p64f) != 0, 0)) {
    const float rho = __builtin_amdgcn_rcpf(st.inv_rho);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int v = 0; v < 16; ++v) st.O[dt][v] *= rho;
    st.l_star *= rho;
    st.inv_rho = 1.0f;
  }
  const float wp = 0.25f * bval * st.inv_rho;      // b_P/4 / rho
  // ---- [O | l] += P^ [V^ | 1]; each V^ group enters two MFMAs (split base),
  // two 32-channel tiles at a time so that consecutive MFMAs are independent.
#pragma unroll
  for (int dp = 0; dp < DT; dp += 2) {
    f16v_t pv[2];
    int vs[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      vs[i] = reinterpret_cast<const int*>(cur + lay.v_scale)[32 * (dp + i) + col];
      const f16v_t c0 = {};
      pv[i] = mfma6_rows<0>(ld_op6(cur + lay.v_op + (size_t)((dp + i) * 2 + 0) * kOpRecord, lane), pop, c0, vs[i]);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
      pv[i] = mfma6_rows<1>(ld_op6(cur + lay.v_op + (size_t)((dp + i) * 2 + 1) * kOpRecord, lane), pop, pv[i],
                            vs[i]);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) st.O[dp + i][v] = __builtin_fmaf(pv[i][v], wp, st.O[dp + i][v]);
  }
  stream_pieces_from<CB>(cs, 7);
  if (NORM == 1) {
    st.l_star = __builtin_fmaf(psum, st.inv_rho, st.l_star);
  } else {
    const f16v_t zero = {};
    const f16v_t lacc = mfma6(ones, pop, zero);
    st.l_star = __builtin_fmaf(lacc[0], wp, st.l_star);
  }
}

template <int G, int NORM, bool DEBUG, bool QMEAN>
__global__ void __launch_bounds__(256, (G == 1 ? 4 : (G == 2 ? 3 : 1))) k_attn_hif4(AttnArgs a, int heads_per_wg, int qsub,
                                                                      int n_qtiles) {
  constexpr int D = 64 * G;
  constexpr int DT = D / 32;
  constexpr ChunkLayout lay = chunk_layout_hif4(G, QMEAN);
  constexpr int cbytes = (int)lay.bytes;
  extern __shared__ __align__(16) uint8_t smem[];
  const TileMap tm = map_tile(a, heads_per_wg, qsub, n_qtiles);
  if (!tm.wg_live) return;
  const int lane = threadIdx.x & 63, h = lane >> 5, col = lane & 31;
  const int qi = tm.qw + col;
  const bool row_ok = tm.active && qi < tm.L;
  const int jw_last = tm.active ? (min(tm.qw + 31, tm.L - 1)) / 64 : -1;
  // the first K/V chunk streams into LDS while the Q tile is quantized
  const uint8_t* ws_base = uniform_ptr(a.ws + ((size_t)(tm.b * a.hkv + tm.hk) * a.NB) * lay.bytes);
  const int wave_u = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  // ---- Q tile: Smooth-QK (fp16(q*s)) then HIF4 into FP6 B operands.  The
  // Q rows and scales are requested before the chunk stream, whose
  // instructions hold the wave while they issue.
  QRaw raw[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const half_t* src = a.q + ((size_t)(tm.t0 + qi) * a.hq + tm.hq) * D + 64 * g + 32 * h;
    const float* sp = a.s ? a.s + (size_t)tm.hk * D + 64 * g + 32 * h : nullptr;
    load_q_half_group(src, sp, row_ok, raw[g]);
  }
  stage_chunk_async<cbytes>(smem, ws_base);
  h2_t xs[G][16];
#pragma unroll
  for (int g = 0; g < G; ++g) smooth_half_group(raw[g], a.s != nullptr, xs[g]);
  float cmu = 0.0f;
  if (QMEAN) cmu = centre_q_row<G>(xs);
  i8_t qop[G];
  float wq[G];
#pragma unroll
  for (int g = 0; g < G; ++g) quantize_q_half_group(xs[g], qop[g], wq[g]);

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

  Hif4State<G> st;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) st.O[dt][v] = 0.0f;
  st.m_run = (half_t)(-__builtin_inff());
  st.l_star = 0.0f;
  st.inv_rho = 1.0f;

  wait_async_copies();
  __syncthreads();

  for (int J = 0; J < tm.nJ; ++J) {
    set_priority_by_work_left(tm.nJ - J);
    const uint8_t* cur = smem + (J & 1) * cbytes;
    // chunk J+1 streams into the other buffer while block J is processed
    const ChunkStream cs{smem + ((J + 1) & 1) * cbytes, ws_base + (size_t)(J + 1 < tm.nJ ? J + 1 : J) * cbytes,
                         wave_u};
    if (J < jw_last)
      hif4_block<G, NORM, DEBUG, QMEAN, false>(a, tm, cur, J, lane, h, col, qi, row_ok, qop, wq, cmu, ones, st, cs);
    else if (J == jw_last)
      hif4_block<G, NORM, DEBUG, QMEAN, true>(a, tm, cur, J, lane, h, col, qi, row_ok, qop, wq, cmu, ones, st, cs);
    else
      stream_pieces_from<cbytes>(cs, 0);
    wait_async_copies();
    __syncthreads();
  }

  // ---- finalize: O = fp16(O*/l*), LSE = m ln2 + ln(l* rho).
  if (row_ok) {
    const float inv = 1.0f / st.l_star;
    half_t* dst = a.o + ((size_t)(tm.t0 + qi) * a.hq + tm.hq) * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        typedef _Float16 h4_t __attribute__((ext_vector_type(4)));
        h4_t o4;
#pragma unroll
        for (int i = 0; i < 4; ++i) o4[i] = (half_t)(st.O[dt][4 * j + i] * inv);
        *reinterpret_cast<h4_t*>(dst + 32 * dt + 8 * j + 4 * h) = o4;
      }
    if (h == 0)
      a.lse[(size_t)tm.hq * a.total_tokens + tm.t0 + qi] =
          (float)st.m_run * 0.69314718055994531f + logf(st.l_star) - logf(st.inv_rho);
  }
}

// ---------------------------------------------------------------------------
// FP16-operand variant (the C16V16 reference): same decomposition, chunk
// stream and softmax as the HiFA4 kernel, 32x32x16 f16 MFMAs, P in fp16 as the
// PV operand, O accumulated by the MFMA, l = rowsum(P).  The two 32-key
// halves of S^T and the D/32 channel tiles of O^T are independent MFMA
// chains, issued interleaved.
template <int D>
__global__ void __launch_bounds__(256, (D <= 128 ? 3 : 1)) k_attn_fp16(AttnArgs a, int heads_per_wg, int qsub, int n_qtiles) {
  constexpr int KC = D / 16;
  constexpr int DT = D / 32;
  constexpr ChunkLayout lay = chunk_layout_fp16(D);
  constexpr int cbytes = (int)lay.bytes;
  constexpr int KB = (int)lay.v_op;               // K operands of a chunk (first part)
  constexpr int VB = cbytes - KB;                 // V operands (second part)
  // whole pieces only, so every wave issues the same number of K pieces and
  // vmcnt(K pieces) leaves only those outstanding
  static_assert(KB % 4096 == 0 && VB % 4096 == 0, "fp16 chunk parts must be whole 4 KiB pieces");
  extern __shared__ __align__(16) uint8_t smem[];
  // K of blocks J and J+1 in two buffers, V of block J in one: V streams in
  // at the start of its block and is waited for just before the PV MFMAs
  uint8_t* kbuf = smem;
  uint8_t* vbuf = smem + 2 * KB;
  const TileMap tm = map_tile(a, heads_per_wg, qsub, n_qtiles);
  if (!tm.wg_live) return;
  const int lane = threadIdx.x & 63, h = lane >> 5, col = lane & 31;
  const int qi = tm.qw + col;
  const bool row_ok = tm.active && qi < tm.L;
  const int jw_last = tm.active ? (min(tm.qw + 31, tm.L - 1)) / 64 : -1;
  const uint8_t* ws_base = uniform_ptr(a.ws + ((size_t)(tm.b * a.hkv + tm.hk) * a.NB) * lay.bytes);
  const int wave_u = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));

  h8_t qf[KC];
#pragma unroll
  for (int kc = 0; kc < KC; ++kc) {
    if (row_ok)
      qf[kc] = *reinterpret_cast<const h8_t*>(a.q + ((size_t)(tm.t0 + qi) * a.hq + tm.hq) * D + 16 * kc + 8 * h);
    else
      for (int e = 0; e < 8; ++e) qf[kc][e] = (half_t)0.0f;
  }
  stream_pieces_from<KB>(ChunkStream{kbuf, ws_base, wave_u}, 0);
  f16v_t O[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) O[dt][v] = 0.0f;
  half_t m_run = (half_t)(-__builtin_inff());
  float l_sum = 0.0f;
  wait_async_copies();
  __syncthreads();

  for (int J = 0; J < tm.nJ; ++J) {
    set_priority_by_work_left(tm.nJ - J);
    const uint8_t* kc_cur = kbuf + (J & 1) * KB;
    const uint8_t* chunkJ = ws_base + (size_t)J * cbytes;
    // V of this block now (its buffer is free since the last block's PV);
    // K of the next block into the other K buffer during the block
    stream_pieces_from<VB>(ChunkStream{vbuf, chunkJ + KB, wave_u}, 0);
    const ChunkStream cs{kbuf + ((J + 1) & 1) * KB, ws_base + (size_t)(J + 1 < tm.nJ ? J + 1 : J) * cbytes, wave_u};
    constexpr int kKPieces = (KB / 16 + 255) / 256;
    if (tm.active && J <= jw_last) {
      f16v_t acc[2] = {};
#pragma unroll
      for (int kc = 0; kc < KC; ++kc)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const h8_t kf = *reinterpret_cast<const h8_t*>(kc_cur + ((size_t)(t * KC + kc) * 64 + lane) * 16);
          acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kf, qf[kc], acc[t], 0, 0, 0);
        }
      stream_piece<KB>(cs, 0);
      h2_t s2[2][8];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int v2 = 0; v2 < 8; ++v2) s2[t][v2] = scale2_to_f16(acc[t][2 * v2], acc[t][2 * v2 + 1], a.c);
      if (64 * J + 63 > tm.qw) {
        const half_t ninf = (half_t)(-__builtin_inff());
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int v = 0; v < 16; ++v)
            if (64 * J + key_of(t, h, v) > qi) s2[t][v >> 1][v & 1] = ninf;
      }
      h2_t mx2 = hmax16(&s2[0][0]);
      mx2 = hmax_halves(max_with_partner(mx2));
      const h2_t mr2 = {m_run, m_run};
      const h2_t mn2 = hmax2(mr2, mx2);
      stream_piece<KB>(cs, 1);
      h2_t p2[2][8];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          h2_t xin[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) xin[i] = s2[t][4 * q + i] - mn2;
          exp2_h2x4(xin, &p2[t][4 * q]);
        }
      float ps = 0.0f;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int v2 = 0; v2 < 8; ++v2) ps = __builtin_amdgcn_fdot2(p2[t][v2], h2_t{(half_t)1, (half_t)1}, ps, false);
      ps = add_with_partner(ps);
      const h2_t rr = exp2_h2(h2_t{(half_t)(mr2[0] - mn2[0]), (half_t)0});
      const float r = (float)rr[0];
      m_run = mn2[0];
      l_sum = l_sum * r + ps;
      stream_pieces_from<KB>(cs, 2);
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
      // V of this block: the wave's own pieces (issued before its K pieces)
      // have landed once at most the K pieces are outstanding; then every
      // wave's share is visible after the barrier
      wait_vmcnt_k<kKPieces>();
      __syncthreads();
#pragma unroll
      for (int c = 0; c < 4; ++c) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const h8_t vf = *reinterpret_cast<const h8_t*>(vbuf + ((size_t)(dt * 4 + c) * 64 + lane) * 16);
          O[dt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vf, pb[c], O[dt], 0, 0, 0);
        }
      }
    } else {
      stream_pieces_from<KB>(cs, 0);
      // the barrier the computing waves take before their PV MFMAs
      wait_vmcnt_k<kKPieces>();
      __syncthreads();
    }
    wait_async_copies();
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
// P-only local operator (the paper's deferred P-only study, Section 4.5 and
// its limitations): Q, K and V stay fp16 and only P is quantized.  Scores and
// the FP16 softmax are those of the FP16-operand kernel; P^ = HIF4(P) as in
// the HiFA4 kernel; the PV product runs on the exact fp16 operand values
// o = u * 2^-sh and an fp32 epilogue applies b_P/4 with the deferred rescale;
// the normalizer accumulates the same P^ (NORM 0) or the pre-quantization P
// (NORM 1).
template <int D, int NORM, bool DEBUG>
__global__ void __launch_bounds__(256, (D <= 128 ? 2 : 1)) k_attn_ponly(AttnArgs a, int heads_per_wg, int qsub,
                                                                       int n_qtiles) {
  constexpr int KC = D / 16;
  constexpr int DT = D / 32;
  constexpr ChunkLayout lay = chunk_layout_fp16(D);
  constexpr int cbytes = (int)lay.bytes;
  extern __shared__ __align__(16) uint8_t smem[];
  const TileMap tm = map_tile(a, heads_per_wg, qsub, n_qtiles);
  if (!tm.wg_live) return;
  const int lane = threadIdx.x & 63, h = lane >> 5, col = lane & 31;
  const int qi = tm.qw + col;
  const bool row_ok = tm.active && qi < tm.L;
  const int jw_last = tm.active ? (min(tm.qw + 31, tm.L - 1)) / 64 : -1;
  const uint8_t* ws_base = uniform_ptr(a.ws + ((size_t)(tm.b * a.hkv + tm.hk) * a.NB) * lay.bytes);
  const int wave_u = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));

  h8_t qf[KC];
#pragma unroll
  for (int kc = 0; kc < KC; ++kc) {
    if (row_ok)
      qf[kc] = *reinterpret_cast<const h8_t*>(a.q + ((size_t)(tm.t0 + qi) * a.hq + tm.hq) * D + 16 * kc + 8 * h);
    else
      for (int e = 0; e < 8; ++e) qf[kc][e] = (half_t)0.0f;
  }
  stage_chunk_async<cbytes>(smem, ws_base);
  f16v_t O[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) O[dt][v] = 0.0f;
  half_t m_run = (half_t)(-__builtin_inff());
  float l_star = 0.0f, inv_rho = 1.0f;
  wait_async_copies();
  __syncthreads();

  for (int J = 0; J < tm.nJ; ++J) {
    const uint8_t* cur = smem + (J & 1) * cbytes;
    const ChunkStream cs{smem + ((J + 1) & 1) * cbytes, ws_base + (size_t)(J + 1 < tm.nJ ? J + 1 : J) * cbytes,
                         wave_u};
    if (tm.active && J <= jw_last) {
      stream_piece<cbytes>(cs, 0);
      f16v_t acc[2] = {};
#pragma unroll
      for (int kc = 0; kc < KC; ++kc)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const h8_t kf = *reinterpret_cast<const h8_t*>(cur + lay.k_op + ((size_t)(t * KC + kc) * 64 + lane) * 16);
          acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kf, qf[kc], acc[t], 0, 0, 0);
        }
      stream_piece<cbytes>(cs, 1);
      h2_t s2[2][8];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int v2 = 0; v2 < 8; ++v2) s2[t][v2] = scale2_to_f16(acc[t][2 * v2], acc[t][2 * v2 + 1], a.c);
      if (64 * J + 63 > tm.qw) {
        const half_t ninf = (half_t)(-__builtin_inff());
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int v = 0; v < 16; ++v)
            if (64 * J + key_of(t, h, v) > qi) s2[t][v >> 1][v & 1] = ninf;
      }
      h2_t mx2 = hmax16(&s2[0][0]);
      mx2 = hmax_halves(max_with_partner(mx2));
      const h2_t mr2 = {m_run, m_run};
      const h2_t mn2 = hmax2(mr2, mx2);
      stream_piece<cbytes>(cs, 2);
      h2_t p2[2][8];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          h2_t xin[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) xin[i] = s2[t][4 * q + i] - mn2;
          exp2_h2x4(xin, &p2[t][4 * q]);
        }
      const h2_t ra = exp2_h2(h2_t{mr2[0], mx2[0]} - mn2);
      const float r = (float)ra[0];
      const float A = (float)ra[1];
      m_run = mn2[0];
      float psum = 0.0f;
      if (NORM == 1) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int v2 = 0; v2 < 8; ++v2)
            psum = __builtin_amdgcn_fdot2(p2[t][v2], h2_t{(half_t)1, (half_t)1}, psum, false);
        psum = add_with_partner(psum);
      }
      stream_piece<cbytes>(cs, 3);
      uint8_t* dcodes = nullptr;
      uint32_t* dmeta = nullptr;
      size_t e;
      if (DEBUG && row_ok && dbg_entry(a, tm.hq, tm.t0 + qi, J, e)) {
        dcodes = a.dbg_codes + e * 32;
        dmeta = a.dbg_meta + e;
      }
      const PQuant pq = quantize_p_block<DEBUG>(p2, A, lane, h, dcodes, dmeta);
      // deferred rescale (as in the HiFA4 kernel): O* = O / rho, l* = l / rho
      if (__builtin_expect(J > 0 && __builtin_amdgcn_ballot_w64(r == 0.0f) != 0, 0)) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int v = 0; v < 16; ++v) O[dt][v] = r == 0.0f ? 0.0f : O[dt][v];
        l_star = r == 0.0f ? 0.0f : l_star;
      }
      inv_rho = (r == 0.0f) ? 1.0f : inv_rho * __builtin_amdgcn_rcpf(r);
      if (__builtin_expect(__builtin_amdgcn_ballot_w64(inv_rho > 0x1p64f) != 0, 0)) {
        const float rho = __builtin_amdgcn_rcpf(inv_rho);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int v = 0; v < 16; ++v) O[dt][v] *= rho;
        l_star *= rho;
        inv_rho = 1.0f;
      }
      const float wp = 0.25f * pq.bval * inv_rho;
      // B operand chunks of the 32x32x16 MFMA: c = 2t + jp holds the values of
      // p2[t][4jp .. 4jp+3], i.e. operand slots 16t + 8jp + [0, 8)
      h8_t pb[4];
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int e = 0; e < 8; ++e) pb[c][e] = pq.ov[8 * c + e];
      if (NORM == 0) {
        float osum = 0.0f;
#pragma unroll
        for (int i = 0; i < 16; ++i)
          osum = __builtin_amdgcn_fdot2(h2_t{pq.ov[2 * i], pq.ov[2 * i + 1]}, h2_t{(half_t)1, (half_t)1}, osum, false);
        l_star = __builtin_fmaf(add_with_partner(osum), wp, l_star);     // sum of P^ (exact before the scale)
      } else {
        l_star = __builtin_fmaf(psum, inv_rho, l_star);
      }
#pragma unroll
      for (int dp = 0; dp < DT; dp += 2) {
        f16v_t pv[2] = {};
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
          for (int i = 0; i < 2; ++i) {
            const h8_t vf =
                *reinterpret_cast<const h8_t*>(cur + lay.v_op + ((size_t)((dp + i) * 4 + c) * 64 + lane) * 16);
            pv[i] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vf, pb[c], pv[i], 0, 0, 0);
          }
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int v = 0; v < 16; ++v) O[dp + i][v] = __builtin_fmaf(pv[i][v], wp, O[dp + i][v]);
        stream_piece<cbytes>(cs, 4 + dp / 2);
      }
      stream_pieces_from<cbytes>(cs, 4 + DT / 2);
    } else {
      stream_pieces_from<cbytes>(cs, 0);
    }
    wait_async_copies();
    __syncthreads();
  }
  if (row_ok) {
    const float inv = 1.0f / l_star;
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
    if (h == 0)
      a.lse[(size_t)tm.hq * a.total_tokens + tm.t0 + qi] =
          (float)m_run * 0.69314718055994531f + logf(l_star) - logf(inv_rho);
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

hipError_t launch_attention(const AttnArgs& a, int norm, int operands, bool qmean, hipStream_t st) {
  if (operands == 2) {
    const size_t lds = 2 * chunk_layout_fp16(a.D).bytes;
    const bool dbg = a.dbg_codes != nullptr;
#define HIFA4_PONLY(D)                                                                                      \
  do {                                                                                                      \
    if (norm == 0)                                                                                          \
      return dbg ? launch_k(k_attn_ponly<D, 0, true>, a, lds, st) : launch_k(k_attn_ponly<D, 0, false>, a, lds, st); \
    return dbg ? launch_k(k_attn_ponly<D, 1, true>, a, lds, st) : launch_k(k_attn_ponly<D, 1, false>, a, lds, st);   \
  } while (0)
    switch (a.D) {
      case 64: HIFA4_PONLY(64);
      case 128: HIFA4_PONLY(128);
      case 256: HIFA4_PONLY(256);
    }
#undef HIFA4_PONLY
    return hipErrorInvalidValue;
  }
  if (operands == 1) {
    const size_t lds = 2 * chunk_layout_fp16(a.D).v_op + (chunk_layout_fp16(a.D).bytes - chunk_layout_fp16(a.D).v_op);
    switch (a.D) {
      case 64: return launch_k(k_attn_fp16<64>, a, lds, st);
      case 128: return launch_k(k_attn_fp16<128>, a, lds, st);
      case 256: return launch_k(k_attn_fp16<256>, a, lds, st);
    }
    return hipErrorInvalidValue;
  }
  const size_t lds = 2 * chunk_layout_hif4(a.D / 64, qmean).bytes;
  const bool dbg = a.dbg_codes != nullptr;
#define HIFA4_DISPATCH_Q(G, QM)                                                                          \
  do {                                                                                                   \
    if (norm == 0)                                                                                       \
      return dbg ? launch_k(k_attn_hif4<G, 0, true, QM>, a, lds, st) : launch_k(k_attn_hif4<G, 0, false, QM>, a, lds, st); \
    return dbg ? launch_k(k_attn_hif4<G, 1, true, QM>, a, lds, st) : launch_k(k_attn_hif4<G, 1, false, QM>, a, lds, st);   \
  } while (0)
#define HIFA4_DISPATCH(G)              \
  do {                                 \
    if (qmean) HIFA4_DISPATCH_Q(G, true); \
    HIFA4_DISPATCH_Q(G, false);        \
  } while (0)
  switch (a.D) {
    case 64: HIFA4_DISPATCH(1);
    case 128: HIFA4_DISPATCH(2);
    case 256: HIFA4_DISPATCH(4);
  }
#undef HIFA4_DISPATCH
#undef HIFA4_DISPATCH_Q
  return hipErrorInvalidValue;
}

}  // namespace hifa4
