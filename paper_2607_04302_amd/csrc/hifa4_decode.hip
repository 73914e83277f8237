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
// decision of the sequential loop:
//   1. scores: per (sequence, kv head, 64-key block) the fp16 scores S2 of the
//      GQA group's query rows, stored, and each row's block maximum;
//   2. splits: each workgroup takes a run of blocks and starts from the
//      running maximum the sequential loop has at its first block (the prefix
//      maximum of the stored block maxima), then applies the FP16 softmax,
//      P^ = HIF4(P) and the PV product as the sequential loop does; it writes
//      its partial O_s and l_s, both relative to the running maximum at its
//      last block;
//   3. merge: O = sum_s O_s R_s and l = sum_s l_s R_s, where R_s is the product
//      of the rescale factors r_J = E(fp16(m_{J-1} - m_J)) of all blocks after
//      split s: the sequential recurrence O <- r_J O + P^_J V^_J unrolled.
// Cache values are decoded to exact fp32 values in LDS: an element is
// +-u 2^-sh b/4 (u <= 7, sh <= 2, b with three significant bits), and every
// product and partial sum of a 64-element group dot of such values is exact in
// fp32, so the scores follow the library's score contract bit for bit.
#include "hifa4_device.h"
#include "hifa4_internal.h"

namespace hifa4 {

namespace {

constexpr int kBlocksPerSplit = 8;
constexpr int kMaxRowsPerWave = 2;   // GQA groups up to 8 query heads per kv head
constexpr int kMaxChPerLane = 4;     // head_dim up to 256

__device__ __forceinline__ int dseq_start(const int* cu, int b, int S) { return cu ? cu[b] : b * S; }
__device__ __forceinline__ int dseq_len(const int* cu, int b, int S) { return cu ? cu[b + 1] - cu[b] : S; }

// Sixteen consecutive elements e0..e0+15 of a canonical group, as exact fp32
// values +-u * 2^-sh * scale (scale = b/4 for the dequantized value, 1 for the
// operand value u * 2^-sh).  w holds the group's code bytes e0/2 .. e0/2+7.
__device__ __forceinline__ void decode16(uint2 w, uint32_t meta, int e0, float scale, float out[16]) {
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const uint32_t word = e < 8 ? w.x : w.y;
    const uint32_t nib = (word >> (4 * (e & 7))) & 15u;
    const int ea = e0 + e;
    const int sh = (int)((meta >> (8 + (ea >> 3))) & 1u) + (int)((meta >> (16 + (ea >> 2))) & 1u);
    const float step = scale * (sh == 0 ? 1.0f : (sh == 1 ? 0.5f : 0.25f));
    const float v = (float)(nib & 7u) * step;
    out[e] = (nib & 8u) ? -v : v;
  }
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
// maximum over aligned groups of `width` lanes (width a power of two <= 64)
__device__ __forceinline__ float group_max(float v, int width) {
  for (int o = width >> 1; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ half_t exp2_h(half_t x) { return exp2_h2(h2_t{x, (half_t)0})[0]; }
__device__ __forceinline__ half_t hmax(half_t a, half_t b) { return a > b ? a : b; }

struct DecodeArgs {
  const uint8_t* qc;       // canonical Q^ of the decode rows [batch, Hq, G, 32]
  const uint32_t* qm;      // [batch, Hq, G]
  const uint8_t* kc;       // canonical K^ cache [tokens, Hkv, G, 32]
  const uint32_t* km;      // [tokens, Hkv, G]
  const uint8_t* vc;       // canonical V^ cache [batch, NB, Hkv, D, 32]
  const uint32_t* vm;      // [batch, NB, Hkv, D]
  const int* cu;
  half_t* s2;              // scores [batch, Hq, NB, 64]
  half_t* mx;              // block maxima [batch, Hq, NB]
  float* opart;            // [batch, Hq, n_split, D]
  float* lpart;            // [batch, Hq, n_split]
  half_t* o;               // [batch, Hq, D]
  float* lse;              // [Hq, batch]
  uint8_t* dbg_codes;      // [Hq, batch, NB, 32] or null
  uint32_t* dbg_meta;      // [Hq, batch, NB]
  int batch, S, NB, hq, hkv, D, n_split;
  float c;
};

// ---------------------------------------------------------------------------
// 1. Scores and block maxima.  Workgroup (J, hk, b), 256 threads.  The query
// rows of the GQA group are kept as operand values and group weights
// w_g = fp32(b_g/4 * c); the block's K^ is decoded one 64-channel group at a
// time into LDS as [channel][key]; wave w owns the rows w and w+4 with
// lane = key, so each lane forms the exact group dot d_g and the accumulator
// acc = fp32(d_0 w_0), then acc = fma(d_g, w_g, acc).
__global__ void __launch_bounds__(256) k_decode_scores(DecodeArgs a) {
  __shared__ float kt[64 * 64];
  __shared__ float qw[8 * 4];
  extern __shared__ float qo[];              // [grp][D]
  const int J = blockIdx.x, hk = blockIdx.y, b = blockIdx.z;
  const int L = dseq_len(a.cu, b, a.S);
  if (64 * J >= L) return;
  const int t0 = dseq_start(a.cu, b, a.S);
  const int D = a.D, G = D >> 6, grp = a.hq / a.hkv;
  const int nk = min(64, L - 64 * J);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int it = tid; it < grp * G * 4; it += 256) {
    const int r = it / (4 * G), g = (it >> 2) % G, qt = it & 3;
    const size_t qi = ((size_t)b * a.hq + hk * grp + r) * G + g;
    const uint32_t meta = a.qm[qi];
    const uint2 w = *reinterpret_cast<const uint2*>(a.qc + qi * 32 + 8 * qt);
    float v[16];
    decode16(w, meta, 16 * qt, 1.0f, v);
#pragma unroll
    for (int e = 0; e < 16; ++e) qo[r * D + 64 * g + 16 * qt + e] = v[e];
    if (qt == 0) qw[r * G + g] = (0.25f * e6m2_value(meta & 255u)) * a.c;
  }
  float acc[kMaxRowsPerWave] = {0.0f, 0.0f};
  for (int g = 0; g < G; ++g) {
    __syncthreads();
    {
      const int key = lane, qt = wave;       // 64 keys x 4 quarters of 16 elements
      float v[16];
      if (key < nk) {
        const size_t gi = ((size_t)(t0 + 64 * J + key) * a.hkv + hk) * G + g;
        const uint32_t meta = a.km[gi];
        const uint2 w = *reinterpret_cast<const uint2*>(a.kc + gi * 32 + 8 * qt);
        decode16(w, meta, 16 * qt, 0.25f * e6m2_value(meta & 255u), v);
      } else {
#pragma unroll
        for (int e = 0; e < 16; ++e) v[e] = 0.0f;
      }
#pragma unroll
      for (int e = 0; e < 16; ++e) kt[(16 * qt + e) * 64 + key] = v[e];
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kMaxRowsPerWave; ++i) {
      const int r = wave + 4 * i;
      if (r >= grp) break;
      const float* qr = qo + r * D + 64 * g;
      float d = 0.0f;                          // exact: every partial sum fits fp32
#pragma unroll 16
      for (int ch = 0; ch < 64; ++ch) d = __builtin_fmaf(qr[ch], kt[ch * 64 + lane], d);
      const float w = qw[r * G + g];
      acc[i] = g == 0 ? d * w : __builtin_fmaf(d, w, acc[i]);
    }
  }
#pragma unroll
  for (int i = 0; i < kMaxRowsPerWave; ++i) {
    const int r = wave + 4 * i;
    if (r >= grp) break;
    const half_t s2 = lane < nk ? (half_t)acc[i] : (half_t)(-__builtin_inff());
    const size_t row = (size_t)b * a.hq + hk * grp + r;
    a.s2[(row * a.NB + J) * 64 + lane] = s2;
    const float m = wave_max((float)s2);
    if (lane == 0) a.mx[row * a.NB + J] = (half_t)m;
  }
}

// ---------------------------------------------------------------------------
// 2. Splits.  Workgroup (split, hk, b), 256 threads: wave w owns the rows w
// and w+4; lane = key for the softmax and P^, lane + 64j = channel for O.
template <int NORM, bool DEBUG>
__global__ void __launch_bounds__(256) k_decode_split(DecodeArgs a) {
  extern __shared__ float dsm[];
  const int sp = blockIdx.x, hk = blockIdx.y, b = blockIdx.z;
  const int L = dseq_len(a.cu, b, a.S);
  const int nblk = (L + 63) >> 6;
  const int J0 = sp * kBlocksPerSplit;
  if (J0 >= nblk) return;
  const int J1 = min(J0 + kBlocksPerSplit, nblk);
  const int D = a.D, grp = a.hq / a.hkv;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  float* vv = dsm;                 // [64 keys][D]
  float* ph = vv + 64 * D;         // [grp][64]
  float O[kMaxRowsPerWave][kMaxChPerLane];
  float l[kMaxRowsPerWave];
  half_t m[kMaxRowsPerWave];
#pragma unroll
  for (int i = 0; i < kMaxRowsPerWave; ++i) {
    l[i] = 0.0f;
#pragma unroll
    for (int j = 0; j < kMaxChPerLane; ++j) O[i][j] = 0.0f;
    const int r = wave + 4 * i;
    float pm = -__builtin_inff();
    if (r < grp) {
      // the running maximum entering block J0: the prefix maximum
      const size_t row = (size_t)b * a.hq + hk * grp + r;
      for (int j = lane; j < J0; j += 64) pm = fmaxf(pm, (float)a.mx[row * a.NB + j]);
      pm = wave_max(pm);
    }
    m[i] = (half_t)pm;
  }
  for (int J = J0; J < J1; ++J) {
    // V^ block: D groups of 64 tokens, decoded into [token][channel]
    for (int it = tid; it < 4 * D; it += 256) {
      const int ch = it % D, qt = it / D;
      const size_t gi = (((size_t)b * a.NB + J) * a.hkv + hk) * D + ch;
      const uint32_t meta = a.vm[gi];
      const uint2 w = *reinterpret_cast<const uint2*>(a.vc + gi * 32 + 8 * qt);
      float v[16];
      decode16(w, meta, 16 * qt, 0.25f * e6m2_value(meta & 255u), v);
#pragma unroll
      for (int e = 0; e < 16; ++e) vv[(16 * qt + e) * D + ch] = v[e];
    }
    float rr[kMaxRowsPerWave];
#pragma unroll
    for (int i = 0; i < kMaxRowsPerWave; ++i) {
      const int r = wave + 4 * i;
      rr[i] = 1.0f;
      if (r >= grp) break;
      const size_t row = (size_t)b * a.hq + hk * grp + r;
      const half_t s2 = a.s2[(row * a.NB + J) * 64 + lane];
      const half_t mn = hmax(m[i], a.mx[row * a.NB + J]);
      const half_t p16 = exp2_h(s2 - mn);     // fp16 difference, then E
      rr[i] = (float)exp2_h(m[i] - mn);
      m[i] = mn;
      // P^ = HIF4(P) over the block's 64 keys (lane = key)
      const float ap = (float)p16;
      const uint32_t base = e6m2_ceil(wave_max(ap));
      const float bval = e6m2_value(base);
      const float a8 = group_max(ap, 8), a4 = group_max(ap, 4);
      const bool e2 = a8 <= 0.875f * bval;
      const bool e3 = a4 <= (e2 ? 0.4375f : 0.875f) * bval;
      const int sh = (int)e2 + (int)e3;
      const float ov = hif4_elem(ap, hif4_rcp_step(base), round_const(sh));   // u * 2^-sh
      ph[r * 64 + lane] = ov * (0.25f * bval);
      const float lsum = wave_sum(NORM == 0 ? ov * (0.25f * bval) : ap);
      l[i] = l[i] * rr[i] + lsum;
      if (DEBUG) {
        const uint32_t u = (uint32_t)(ov * (float)(1 << sh));
        const uint32_t hi = (uint32_t)__shfl_xor((int)u, 1);
        const size_t dj = ((size_t)(hk * grp + r) * a.batch + b) * a.NB + J;
        if ((lane & 1) == 0) a.dbg_codes[dj * 32 + (lane >> 1)] = (uint8_t)(u | (hi << 4));
        const uint64_t b2 = __ballot(e2), b3 = __ballot(e3);
        if (lane == 0) {
          uint32_t w2 = 0, w3 = 0;
          for (int k = 0; k < 8; ++k) w2 |= (uint32_t)((b2 >> (8 * k)) & 1u) << k;
          for (int q = 0; q < 16; ++q) w3 |= (uint32_t)((b3 >> (4 * q)) & 1u) << q;
          a.dbg_meta[dj] = base | (w2 << 8) | (w3 << 16);
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kMaxRowsPerWave; ++i) {
      const int r = wave + 4 * i;
      if (r >= grp) break;
      const float* pr = ph + r * 64;
#pragma unroll
      for (int j = 0; j < kMaxChPerLane; ++j) {
        if (64 * j >= D) break;
        const int ch = lane + 64 * j;
        float acc = 0.0f;
#pragma unroll 16
        for (int key = 0; key < 64; ++key) acc = __builtin_fmaf(pr[key], vv[key * D + ch], acc);
        O[i][j] = __builtin_fmaf(O[i][j], rr[i], acc);
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < kMaxRowsPerWave; ++i) {
    const int r = wave + 4 * i;
    if (r >= grp) break;
    const size_t row = (size_t)b * a.hq + hk * grp + r;
    float* dst = a.opart + (row * a.n_split + sp) * D;
#pragma unroll
    for (int j = 0; j < kMaxChPerLane; ++j)
      if (64 * j < D) dst[lane + 64 * j] = O[i][j];
    if (lane == 0) a.lpart[row * a.n_split + sp] = l[i];
  }
}

// ---------------------------------------------------------------------------
// 3. Merge.  One wave per row (b, query head).  A forward pass over the block
// maxima, 64 blocks at a time, gives the running maxima m_J (prefix maxima),
// the factors r_J = E(fp16(m_{J-1} - m_J)) and their product over each split;
// a backward pass over the splits turns those into R_s = the product over
// all later splits.
__global__ void __launch_bounds__(64) k_decode_merge(DecodeArgs a) {
  extern __shared__ float R[];                    // [n_split]
  const int row = blockIdx.x;                     // b * hq + head
  const int b = row / a.hq, head = row % a.hq;
  const int L = dseq_len(a.cu, b, a.S);
  const int nblk = (L + 63) >> 6;
  if (nblk == 0) return;
  const int ns = (nblk + kBlocksPerSplit - 1) / kBlocksPerSplit;
  const int lane = threadIdx.x;
  half_t carry = (half_t)(-__builtin_inff());
  for (int J0 = 0; J0 < nblk; J0 += 64) {
    const int J = J0 + lane;
    float f = J < nblk ? (float)a.mx[(size_t)row * a.NB + J] : -__builtin_inff();
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const float t = __shfl_up(f, o);
      if (lane >= o) f = fmaxf(f, t);
    }
    const half_t incl = hmax((half_t)f, carry);
    const float prevf = __shfl_up((float)incl, 1);
    const half_t prev = lane == 0 ? carry : (half_t)prevf;
    float p = J < nblk ? (float)exp2_h(prev - incl) : 1.0f;
    p *= __shfl_xor(p, 1);
    p *= __shfl_xor(p, 2);
    p *= __shfl_xor(p, 4);
    const int s = (J0 >> 3) + (lane >> 3);
    if ((lane & 7) == 0 && s < ns) R[s] = p;
    carry = (half_t)__shfl((float)incl, 63);
  }
  __syncthreads();
  float tail = 1.0f;
  for (int s1 = ns; s1 > 0; s1 -= 64) {
    const int s = s1 - 1 - lane;
    const float v = s >= 0 ? R[s] : 1.0f;
    float incl = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const float t = __shfl_up(incl, o);
      if (lane >= o) incl *= t;
    }
    const float excl = __shfl_up(incl, 1);
    if (s >= 0) R[s] = tail * (lane == 0 ? 1.0f : excl);
    tail *= __shfl(incl, 63);
  }
  __syncthreads();
  float lacc = 0.0f;
  for (int s = lane; s < ns; s += 64) lacc = __builtin_fmaf(a.lpart[(size_t)row * a.n_split + s], R[s], lacc);
  const float lsum = wave_sum(lacc);
  const float inv = 1.0f / lsum;
  for (int ch = lane; ch < a.D; ch += 64) {
    float acc = 0.0f;
    for (int s = 0; s < ns; ++s) acc = __builtin_fmaf(a.opart[((size_t)row * a.n_split + s) * a.D + ch], R[s], acc);
    a.o[(size_t)row * a.D + ch] = (half_t)(acc * inv);
  }
  if (lane == 0) a.lse[(size_t)head * a.batch + b] = (float)carry * 0.69314718055994531f + logf(lsum);
}

void decode_offsets(int batch, int hq, int D, int NB, size_t off[7]) {
  const int G = D / 64;
  const int n_split = (NB + kBlocksPerSplit - 1) / kBlocksPerSplit;
  size_t o = 0;
  off[0] = o; o += round_up256((size_t)batch * hq * G * 32);                 // Q^ codes
  off[1] = o; o += round_up256((size_t)batch * hq * G * 4);                  // Q^ metadata
  off[2] = o; o += round_up256((size_t)batch * hq * NB * 64 * 2);            // scores
  off[3] = o; o += round_up256((size_t)batch * hq * NB * 2);                 // block maxima
  off[4] = o; o += round_up256((size_t)batch * hq * n_split * D * 4);        // partial O
  off[5] = o; o += round_up256((size_t)batch * hq * n_split * 4);            // partial l
  off[6] = o;
}

template <typename K>
hipError_t allow_lds(K kern, size_t bytes) {
  if (bytes <= 65536) return hipSuccess;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)bytes);
}

}  // namespace

size_t decode_workspace_bytes(int batch, int hq, int D, int NB) {
  size_t off[7];
  decode_offsets(batch, hq, D, NB, off);
  return off[6];
}

hipError_t launch_decode(const DecodeLaunch& d, hipStream_t st) {
  size_t off[7];
  decode_offsets(d.batch, d.hq, d.D, d.NB, off);
  uint8_t* ws = d.ws;
  DecodeArgs a;
  a.qc = ws + off[0];
  a.qm = reinterpret_cast<const uint32_t*>(ws + off[1]);
  a.kc = d.kc;
  a.km = d.km;
  a.vc = d.vc;
  a.vm = d.vm;
  a.cu = d.cu;
  a.s2 = reinterpret_cast<half_t*>(ws + off[2]);
  a.mx = reinterpret_cast<half_t*>(ws + off[3]);
  a.opart = reinterpret_cast<float*>(ws + off[4]);
  a.lpart = reinterpret_cast<float*>(ws + off[5]);
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
  a.n_split = (d.NB + kBlocksPerSplit - 1) / kBlocksPerSplit;
  a.c = d.c;
  const int grp = d.hq / d.hkv;
  hipError_t e = launch_quant_rows(d.q, d.s, ws + off[0], reinterpret_cast<uint32_t*>(ws + off[1]), d.batch, d.hq,
                                   d.hkv, d.D, false, st);
  if (e != hipSuccess) return e;
  const size_t lds1 = (size_t)grp * d.D * sizeof(float);
  k_decode_scores<<<dim3(d.NB, d.hkv, d.batch), dim3(256), lds1, st>>>(a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (d.ev && (e = hipEventRecord(d.ev[1], st)) != hipSuccess) return e;
  const size_t lds2 = ((size_t)64 * d.D + (size_t)grp * 64) * sizeof(float);
  const dim3 g2(a.n_split, d.hkv, d.batch);
  if (d.norm == 0) {
    if (d.dbg_codes) {
      if ((e = allow_lds(k_decode_split<0, true>, lds2)) != hipSuccess) return e;
      k_decode_split<0, true><<<g2, dim3(256), lds2, st>>>(a);
    } else {
      if ((e = allow_lds(k_decode_split<0, false>, lds2)) != hipSuccess) return e;
      k_decode_split<0, false><<<g2, dim3(256), lds2, st>>>(a);
    }
  } else {
    if (d.dbg_codes) {
      if ((e = allow_lds(k_decode_split<1, true>, lds2)) != hipSuccess) return e;
      k_decode_split<1, true><<<g2, dim3(256), lds2, st>>>(a);
    } else {
      if ((e = allow_lds(k_decode_split<1, false>, lds2)) != hipSuccess) return e;
      k_decode_split<1, false><<<g2, dim3(256), lds2, st>>>(a);
    }
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  k_decode_merge<<<dim3(d.batch * d.hq), dim3(64), (size_t)a.n_split * sizeof(float), st>>>(a);
  return hipGetLastError();
}

}  // namespace hifa4
