// Issue cost of the instruction types the attention kernels are made of, on
// one MI355X (gfx950): each kernel runs 8 independent chains of one
// instruction per lane (16 rounds unrolled per loop iteration) in 4096
// workgroups of 256 threads (16 waves per SIMD), and the cost is the kernel
// time x 1024 SIMDs / wave64 instructions issued.  Prints one JSON line per
// instruction.  A measurement tool for the roofline of bench.py; the library
// does not use it.
#include <hip/hip_runtime.h>

#include <cstdio>

typedef int i8v __attribute__((ext_vector_type(8)));
typedef int i6v __attribute__((ext_vector_type(6)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef _Float16 h32v __attribute__((ext_vector_type(32)));
typedef _Float16 h8v __attribute__((ext_vector_type(8)));

constexpr int kChains = 8;
constexpr int kRounds = 16;

#define VALU_KERNEL(NAME, ASM)                                                                   \
  __global__ void __launch_bounds__(256) NAME(const unsigned* in, unsigned* out, int iters) {     \
    unsigned a[kChains];                                                                         \
    const unsigned b = in[threadIdx.x & 63], c = in[64 + (threadIdx.x & 63)];                   \
    for (int i = 0; i < kChains; ++i) a[i] = in[128 + i] ^ threadIdx.x;                         \
    for (int it = 0; it < iters; ++it) {                                                         \
      _Pragma("unroll") for (int r = 0; r < kRounds; ++r) {                                     \
        _Pragma("unroll") for (int i = 0; i < kChains; ++i)                                     \
          asm volatile(ASM : "+v"(a[i]) : "v"(b), "v"(c) : "s10", "s11", "vcc");               \
      }                                                                                          \
    }                                                                                            \
    unsigned s = 0;                                                                              \
    for (int i = 0; i < kChains; ++i) s ^= a[i];                                                 \
    out[blockIdx.x * blockDim.x + threadIdx.x] = s;                                              \
  }

VALU_KERNEL(k_fma_f32, "v_fma_f32 %0, %0, %1, %2")
VALU_KERNEL(k_mul_f32, "v_mul_f32 %0, %0, %1")
VALU_KERNEL(k_add_f32, "v_add_f32 %0, %0, %1")
VALU_KERNEL(k_mov_b32, "v_mov_b32 %0, %1")
VALU_KERNEL(k_add_u32, "v_add_u32 %0, %0, %1")
VALU_KERNEL(k_max_f32, "v_max_f32 %0, %0, %1")
VALU_KERNEL(k_pk_fma_f16, "v_pk_fma_f16 %0, %0, %1, %2")
VALU_KERNEL(k_pk_max_f16, "v_pk_max_f16 %0, %0, %1")
VALU_KERNEL(k_pk_add_f16, "v_pk_add_f16 %0, %0, %1")
VALU_KERNEL(k_pk_sub_u16, "v_pk_sub_u16 %0, %0, %1")
VALU_KERNEL(k_max_f16_sdwa, "v_max_f16_sdwa %0, %0, %1 dst_sel:WORD_1 dst_unused:UNUSED_PRESERVE src0_sel:WORD_1 src1_sel:WORD_0")
VALU_KERNEL(k_cvt_pk_f16_f32, "v_cvt_pk_f16_f32 %0, %0, %1")
VALU_KERNEL(k_cvt_f32_f16, "v_cvt_f32_f16 %0, %0")
VALU_KERNEL(k_perm_b32, "v_perm_b32 %0, %0, %1, %2")
VALU_KERNEL(k_bfe_u32, "v_bfe_u32 %0, %0, %1, %2")
VALU_KERNEL(k_cmp_cndmask, "v_cmp_gt_u32 s[10:11], %1, %2\n\tv_cndmask_b32 %0, %0, %1, s[10:11]")
VALU_KERNEL(k_fma_mix_f32, "v_fma_mix_f32 %0, %0, %1, %2 op_sel_hi:[1,0,0]")
VALU_KERNEL(k_fma_mixlo_f16, "v_fma_mixlo_f16 %0, %0, %1, %2 op_sel_hi:[1,0,1]")
VALU_KERNEL(k_exp_f16, "v_exp_f16 %0, %0")
VALU_KERNEL(k_exp_f32, "v_exp_f32 %0, %0")
VALU_KERNEL(k_rcp_f32, "v_rcp_f32 %0, %0")
VALU_KERNEL(k_permlane32_swap, "v_permlane32_swap_b32 %0, %1")

// 64-bit address arithmetic (the form the compiler emits for global
// addresses built from a per-lane base and a uniform offset)
__global__ void __launch_bounds__(256) k_lshl_add_u64(const unsigned* in, unsigned* out, int iters) {
  unsigned long long a[kChains];
  const unsigned long long b =
      ((unsigned long long)in[threadIdx.x & 63] << 32) | (unsigned long long)in[64 + (threadIdx.x & 63)];
  for (int i = 0; i < kChains; ++i) a[i] = in[128 + i] ^ threadIdx.x;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
#pragma unroll
      for (int i = 0; i < kChains; ++i) asm volatile("v_lshl_add_u64 %0, %0, 0, %1" : "+v"(a[i]) : "v"(b));
    }
  }
  unsigned s = 0;
  for (int i = 0; i < kChains; ++i) s ^= (unsigned)a[i] ^ (unsigned)(a[i] >> 32);
  out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

constexpr int kMfmaChains = 4;
__global__ void __launch_bounds__(256) k_mfma_fp6(const unsigned* in, unsigned* out, int iters) {
  i8v a, b;
  for (int i = 0; i < 8; ++i) {
    a[i] = (int)(in[i] ^ threadIdx.x);
    b[i] = (int)in[8 + i];
  }
  a[6] = a[7] = b[6] = b[7] = 0;
  f16v c[kMfmaChains];
  for (int k = 0; k < kMfmaChains; ++k)
    for (int i = 0; i < 16; ++i) c[k][i] = 0.f;
  for (int it = 0; it < iters; ++it)
#pragma unroll
    for (int k = 0; k < kMfmaChains; ++k)
      c[k] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c[k], 2, 2, 0, 127, 0, 127);
  float s = 0;
  for (int k = 0; k < kMfmaChains; ++k)
    for (int i = 0; i < 16; ++i) s += c[k][i];
  out[blockIdx.x * blockDim.x + threadIdx.x] = __float_as_uint(s);
}

__global__ void __launch_bounds__(256) k_mfma_f16(const unsigned* in, unsigned* out, int iters) {
  h8v a, b;
  for (int i = 0; i < 8; ++i) {
    a[i] = (_Float16)(float)(in[i] & 7);
    b[i] = (_Float16)(float)(in[8 + i] & 3);
  }
  f16v c[kMfmaChains];
  for (int k = 0; k < kMfmaChains; ++k)
    for (int i = 0; i < 16; ++i) c[k][i] = 0.f;
  for (int it = 0; it < iters; ++it)
#pragma unroll
    for (int k = 0; k < kMfmaChains; ++k) c[k] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c[k], 0, 0, 0);
  float s = 0;
  for (int k = 0; k < kMfmaChains; ++k)
    for (int i = 0; i < 16; ++i) s += c[k][i];
  out[blockIdx.x * blockDim.x + threadIdx.x] = __float_as_uint(s);
}

__global__ void __launch_bounds__(256) k_cvt_pk32_fp6_f16(const unsigned* in, unsigned* out, int iters) {
  h32v x;
  for (int i = 0; i < 32; ++i) x[i] = (_Float16)((float)(in[i] & 7) * 0.25f);
  int acc = 0;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const i6v y = __builtin_amdgcn_cvt_scalef32_pk32_fp6_f16(x, 1.0f + (float)r);
      acc ^= y[0] ^ y[5];
      x[0] = (_Float16)(float)(y[1] & 3);
    }
  }
  out[blockIdx.x * blockDim.x + threadIdx.x] = (unsigned)acc;
}

typedef void (*Kernel)(const unsigned*, unsigned*, int);

int main() {
  const int blocks = 256 * 16, threads = 256;
  unsigned *in = nullptr, *out = nullptr;
  if (hipMalloc(&in, 4096) != hipSuccess || hipMalloc(&out, (size_t)blocks * threads * 4) != hipSuccess) return 1;
  unsigned h[1024];
  for (int i = 0; i < 1024; ++i) h[i] = 0x3c003c00u ^ (unsigned)(i * 7);
  if (hipMemcpy(in, h, sizeof h, hipMemcpyHostToDevice) != hipSuccess) return 1;
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return 1;
  struct Case {
    const char* name;
    Kernel k;
    int iters;
    double insts_per_iter;   // per wave and loop iteration
  };
  const double v = kChains * kRounds;
  const Case cases[] = {
      {"v_fma_f32", k_fma_f32, 400, v}, {"v_mul_f32", k_mul_f32, 400, v}, {"v_add_f32", k_add_f32, 400, v},
      {"v_mov_b32", k_mov_b32, 400, v}, {"v_add_u32", k_add_u32, 400, v}, {"v_max_f32", k_max_f32, 400, v},
      {"v_pk_fma_f16", k_pk_fma_f16, 400, v}, {"v_pk_max_f16", k_pk_max_f16, 400, v},
      {"v_pk_add_f16", k_pk_add_f16, 400, v}, {"v_pk_sub_u16", k_pk_sub_u16, 400, v},
      {"v_max_f16_sdwa", k_max_f16_sdwa, 400, v}, {"v_cvt_pk_f16_f32", k_cvt_pk_f16_f32, 400, v},
      {"v_cvt_f32_f16", k_cvt_f32_f16, 400, v}, {"v_perm_b32", k_perm_b32, 400, v}, {"v_bfe_u32", k_bfe_u32, 400, v},
      {"v_cmp_gt_u32+v_cndmask_b32", k_cmp_cndmask, 400, v}, {"v_fma_mix_f32", k_fma_mix_f32, 400, v},
      {"v_fma_mixlo_f16", k_fma_mixlo_f16, 400, v}, {"v_exp_f16", k_exp_f16, 400, v}, {"v_exp_f32", k_exp_f32, 400, v},
      {"v_rcp_f32", k_rcp_f32, 400, v}, {"v_permlane32_swap_b32", k_permlane32_swap, 400, v},
      {"v_lshl_add_u64", k_lshl_add_u64, 400, v},
      {"v_mfma_scale_f32_32x32x64_f8f6f4 (fp6)", k_mfma_fp6, 200, kMfmaChains},
      {"v_mfma_f32_32x32x16_f16", k_mfma_f16, 200, kMfmaChains},
      {"v_cvt_scalef32_pk32_fp6_f16", k_cvt_pk32_fp6_f16, 200, 8}};
  for (const Case& c : cases) {
    float best = 1e30f;
    for (int rep = 0; rep < 4; ++rep) {
      if (hipEventRecord(e0) != hipSuccess) return 1;
      c.k<<<blocks, threads>>>(in, out, c.iters);
      if (hipGetLastError() != hipSuccess) return 1;
      if (hipEventRecord(e1) != hipSuccess || hipEventSynchronize(e1) != hipSuccess) return 1;
      float ms = 0;
      if (hipEventElapsedTime(&ms, e0, e1) != hipSuccess) return 1;
      if (ms < best) best = ms;
    }
    const double waves = (double)blocks * threads / 64;
    const double ns = best * 1e6 * 1024 / (waves * c.iters * c.insts_per_iter);
    printf("{\"instruction\": \"%s\", \"ns_per_wave64_per_simd\": %.3f, \"cycles_at_2.4GHz\": %.2f}\n", c.name, ns,
           ns * 2.4);
  }
  return 0;
}
