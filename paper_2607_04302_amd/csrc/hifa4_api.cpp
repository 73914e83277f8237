// C ABI of libhifa4 (declared in include/hifa4.h): argument validation,
// workspace carving, kernel launches and the host side of calibration.
#include "../../include/hifa4.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <initializer_list>
#include <mutex>
#include <string>
#include <vector>

#include "hifa4_decode.h"
#include "hifa4_internal.h"

namespace {

thread_local std::string g_last_error;

hifa4_status fail(hifa4_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
hifa4_status fail(hifa4_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

hifa4_status hip_fail(hipError_t e, const char* what) {
  return fail(HIFA4_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

struct Dims {
  long tokens;   // rows of the [T, H, D] view
  int S;         // max_seqlen
  int NB;        // ceil(S/64)
};

// Vector loads and stores of the kernels need these alignments (a pointer
// that may be NULL passes).
bool aligned(const void* ptr, uintptr_t a) { return ((uintptr_t)ptr % a) == 0; }

hifa4_status check_aligned16(std::initializer_list<const void*> ptrs) {
  for (const void* ptr : ptrs)
    if (!aligned(ptr, 16)) return fail(HIFA4_ERR_INVALID_ARGUMENT, "tensor pointer %p is not 16-byte aligned", ptr);
  return HIFA4_OK;
}

hifa4_status check_aligned4(std::initializer_list<const void*> ptrs) {
  for (const void* ptr : ptrs)
    if (!aligned(ptr, 4)) return fail(HIFA4_ERR_INVALID_ARGUMENT, "pointer %p is not 4-byte aligned", ptr);
  return HIFA4_OK;
}

hifa4_status check_problem(const hifa4_problem* p, Dims* d) {
  if (!p) return fail(HIFA4_ERR_INVALID_ARGUMENT, "problem is NULL");
  if (p->batch <= 0 || p->num_heads_q <= 0 || p->num_heads_kv <= 0 || p->max_seqlen < 0)
    return fail(HIFA4_ERR_INVALID_ARGUMENT, "batch, head counts must be > 0 and max_seqlen >= 0");
  if (p->num_heads_q % p->num_heads_kv != 0)
    return fail(HIFA4_ERR_UNSUPPORTED, "num_heads_q (%d) must be a multiple of num_heads_kv (%d)", p->num_heads_q,
                p->num_heads_kv);
  if (p->head_dim != 64 && p->head_dim != 128 && p->head_dim != 256)
    return fail(HIFA4_ERR_UNSUPPORTED, "head_dim %d not in {64, 128, 256}", p->head_dim);
  if (p->causal != 1) return fail(HIFA4_ERR_UNSUPPORTED, "only causal prefill (causal = 1) is supported");
  if (p->cu_seqlens && p->total_tokens < 0) return fail(HIFA4_ERR_INVALID_ARGUMENT, "total_tokens < 0");
  d->S = p->max_seqlen;
  d->NB = (p->max_seqlen + 63) / 64;
  d->tokens = p->cu_seqlens ? (long)p->total_tokens : (long)p->batch * p->max_seqlen;
  if (d->tokens > (1L << 31) / std::max(1, p->num_heads_q))
    return fail(HIFA4_ERR_UNSUPPORTED, "problem too large for 32-bit row indexing");
  return HIFA4_OK;
}

}  // namespace

extern "C" {

const char* hifa4_last_error(void) { return g_last_error.c_str(); }

size_t hifa4_workspace_bytes(const hifa4_problem* p, const hifa4_fwd_options* opt) {
  Dims d;
  if (check_problem(p, &d) != HIFA4_OK) return 0;
  const bool fp16 = opt && (opt->operands == HIFA4_OPERANDS_FP16 || opt->operands == HIFA4_OPERANDS_P_ONLY);
  const bool qmean = opt && opt->q_mean != 0;
  const size_t chunk = fp16 ? hifa4::chunk_layout_fp16(p->head_dim).bytes
                            : hifa4::chunk_layout_hif4(p->head_dim / 64, qmean).bytes;
  return chunk * (size_t)p->batch * p->num_heads_kv * std::max(1, d.NB);
}

size_t hifa4_calibrate_workspace_bytes(const hifa4_problem* p, int32_t n_calib) {
  if (!p || n_calib <= 0 || p->num_heads_kv <= 0 || p->head_dim <= 0) return 0;
  return hifa4::round_up256((size_t)n_calib * 2 * p->num_heads_kv * p->head_dim * 4) + 32768 * 8;
}

hifa4_status hifa4_quantize_qk(const hifa4_problem* p, const void* q, const void* k, const float* s, void* q_codes,
                               void* q_meta, void* k_codes, void* k_meta, void* stream) {
  Dims d;
  hifa4_status st = check_problem(p, &d);
  if (st != HIFA4_OK) return st;
  const bool q_none = !q && !q_codes && !q_meta;
  if ((!q_none && (!q || !q_codes || !q_meta)) || !k || !k_codes || !k_meta)
    return fail(HIFA4_ERR_INVALID_ARGUMENT, "null tensor pointer");
  if ((st = check_aligned16({q, k, s, q_codes, k_codes})) != HIFA4_OK) return st;
  if ((st = check_aligned4({q_meta, k_meta, p->cu_seqlens})) != HIFA4_OK) return st;
  hipStream_t hs = (hipStream_t)stream;
  using hifa4::half_t;
  hipError_t e = hipSuccess;
  if (!q_none) {
    e = hifa4::launch_quant_rows((const half_t*)q, s, (uint8_t*)q_codes, (uint32_t*)q_meta, d.tokens,
                                 p->num_heads_q, p->num_heads_kv, p->head_dim, false, hs);
    if (e != hipSuccess) return hip_fail(e, "quantize Q");
  }
  e = hifa4::launch_quant_rows((const half_t*)k, s, (uint8_t*)k_codes, (uint32_t*)k_meta, d.tokens, p->num_heads_kv,
                               p->num_heads_kv, p->head_dim, true, hs);
  if (e != hipSuccess) return hip_fail(e, "quantize K");
  return HIFA4_OK;
}

hifa4_status hifa4_quantize_v(const hifa4_problem* p, const void* v, void* v_codes, void* v_meta, void* stream) {
  Dims d;
  hifa4_status st = check_problem(p, &d);
  if (st != HIFA4_OK) return st;
  if (!v || !v_codes || !v_meta) return fail(HIFA4_ERR_INVALID_ARGUMENT, "null tensor pointer");
  if ((st = check_aligned16({v, v_codes})) != HIFA4_OK) return st;
  if ((st = check_aligned4({v_meta, p->cu_seqlens})) != HIFA4_OK) return st;
  hipError_t e = hifa4::launch_quant_v((const hifa4::half_t*)v, p->cu_seqlens, (uint8_t*)v_codes, (uint32_t*)v_meta,
                                       p->batch, d.S, d.NB, p->num_heads_kv, p->head_dim, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "quantize V");
  return HIFA4_OK;
}

hifa4_status hifa4_attention_fwd(const hifa4_problem* p, const hifa4_fwd_options* opt, const void* q, const void* k,
                                 const void* v, const float* s, void* o, float* lse, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  Dims d;
  hifa4_status st = check_problem(p, &d);
  if (st != HIFA4_OK) return st;
  if (!opt) return fail(HIFA4_ERR_INVALID_ARGUMENT, "options is NULL");
  if (opt->norm != HIFA4_NORM_PREORDER && opt->norm != HIFA4_NORM_INCONSISTENT)
    return fail(HIFA4_ERR_INVALID_ARGUMENT, "unknown norm %d", opt->norm);
  if (opt->operands != HIFA4_OPERANDS_HIF4 && opt->operands != HIFA4_OPERANDS_FP16 &&
      opt->operands != HIFA4_OPERANDS_P_ONLY)
    return fail(HIFA4_ERR_INVALID_ARGUMENT, "unknown operands %d", opt->operands);
  if (!q || !k || !v || !o || !lse) return fail(HIFA4_ERR_INVALID_ARGUMENT, "null tensor pointer");
  if ((opt->debug_p_codes == nullptr) != (opt->debug_p_meta == nullptr))
    return fail(HIFA4_ERR_INVALID_ARGUMENT, "debug_p_codes and debug_p_meta must both be set or both be NULL");
  if ((st = check_aligned16({q, k, v, o, s, workspace, opt->debug_p_codes})) != HIFA4_OK) return st;
  if ((st = check_aligned4({lse, p->cu_seqlens, opt->debug_p_meta})) != HIFA4_OK) return st;
  if (opt->debug_head_count < 0 || opt->debug_token_count < 0 || opt->debug_head_begin < 0 ||
      opt->debug_token_begin < 0 || (!opt->debug_head_count && opt->debug_head_begin) ||
      (!opt->debug_token_count && opt->debug_token_begin) ||
      (long)opt->debug_head_begin + opt->debug_head_count > p->num_heads_q ||
      (long)opt->debug_token_begin + opt->debug_token_count > (long)d.tokens)
    return fail(HIFA4_ERR_INVALID_ARGUMENT, "debug window outside the problem");
  // FP16 and P-only keep Q, K and V in fp16 (fp16 chunk layout, no smoothing)
  const bool fp16 = opt->operands != HIFA4_OPERANDS_HIF4;
  if (fp16 && opt->q_mean)
    return fail(HIFA4_ERR_UNSUPPORTED, "q_mean applies to HIF4 operands only");
  const bool qmean = opt->q_mean != 0;
  const float* sm = (!fp16 && opt->smooth_qk) ? s : nullptr;
  if (!fp16 && opt->smooth_qk && !s) return fail(HIFA4_ERR_INVALID_ARGUMENT, "smooth_qk set but s is NULL");
  if (d.tokens == 0 || d.S == 0) return HIFA4_OK;
  const size_t need = hifa4_workspace_bytes(p, opt);
  if (!workspace || workspace_bytes < need)
    return fail(HIFA4_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", workspace_bytes, need);
  hipStream_t hs = (hipStream_t)stream;
  hipEvent_t* ev = (hipEvent_t*)opt->timing_events;
  hipError_t e = hipSuccess;
  if (ev && (e = hipEventRecord(ev[0], hs)) != hipSuccess) return hip_fail(e, "timing event");
  e = hifa4::launch_prep_kv((const hifa4::half_t*)k, (const hifa4::half_t*)v, sm, p->cu_seqlens, (uint8_t*)workspace,
                            p->batch, d.S, d.NB, p->num_heads_kv, p->head_dim, fp16, qmean, hs);
  if (e != hipSuccess) return hip_fail(e, "K/V pre-pass");
  if (ev && (e = hipEventRecord(ev[1], hs)) != hipSuccess) return hip_fail(e, "timing event");
  hifa4::AttnArgs a;
  a.q = (const hifa4::half_t*)q;
  a.s = sm;
  a.cu = p->cu_seqlens;
  a.ws = (const uint8_t*)workspace;
  a.o = (hifa4::half_t*)o;
  a.lse = lse;
  const bool dump = opt->operands != HIFA4_OPERANDS_FP16;
  a.dbg_codes = dump ? (uint8_t*)opt->debug_p_codes : nullptr;
  a.dbg_meta = dump ? (uint32_t*)opt->debug_p_meta : nullptr;
  a.dbg_h0 = opt->debug_head_count ? opt->debug_head_begin : 0;
  a.dbg_nh = opt->debug_head_count ? opt->debug_head_count : p->num_heads_q;
  a.dbg_t0 = opt->debug_token_count ? opt->debug_token_begin : 0;
  a.dbg_nt = opt->debug_token_count ? opt->debug_token_count : (int)d.tokens;
  a.batch = p->batch;
  a.S = d.S;
  a.NB = d.NB;
  a.hq = p->num_heads_q;
  a.hkv = p->num_heads_kv;
  a.D = p->head_dim;
  a.total_tokens = (int)d.tokens;
  a.c = (float)(1.4426950408889634 / std::sqrt((double)p->head_dim));
  e = hifa4::launch_attention(a, opt->norm, opt->operands, qmean, hs);
  if (e != hipSuccess) return hip_fail(e, "attention kernel");
  if (ev && (e = hipEventRecord(ev[2], hs)) != hipSuccess) return hip_fail(e, "timing event");
  return HIFA4_OK;
}

size_t hifa4_decode_workspace_bytes(const hifa4_problem* p) {
  Dims d;
  if (check_problem(p, &d) != HIFA4_OK) return 0;
  return hifa4::decode_workspace_bytes(p->batch, p->num_heads_q, p->num_heads_kv, p->head_dim, std::max(1, d.NB));
}

hifa4_status hifa4_decode_fwd(const hifa4_problem* p, const hifa4_fwd_options* opt, const void* q,
                              const void* k_codes, const void* k_meta, const void* v_codes, const void* v_meta,
                              const float* s, void* o, float* lse, void* workspace, size_t workspace_bytes,
                              void* stream) {
  Dims d;
  hifa4_status st = check_problem(p, &d);
  if (st != HIFA4_OK) return st;
  if (!opt) return fail(HIFA4_ERR_INVALID_ARGUMENT, "options is NULL");
  if (opt->norm != HIFA4_NORM_PREORDER && opt->norm != HIFA4_NORM_INCONSISTENT)
    return fail(HIFA4_ERR_INVALID_ARGUMENT, "unknown norm %d", opt->norm);
  if (opt->operands != HIFA4_OPERANDS_HIF4)
    return fail(HIFA4_ERR_UNSUPPORTED, "decode reads a HIF4 cache: operands must be HIFA4_OPERANDS_HIF4");
  if (opt->q_mean) return fail(HIFA4_ERR_UNSUPPORTED, "q_mean is not supported by decode (the cache has no key sums)");
  if (p->num_heads_q / p->num_heads_kv > 8)
    return fail(HIFA4_ERR_UNSUPPORTED, "decode supports at most 8 query heads per kv head (got %d)",
                p->num_heads_q / p->num_heads_kv);
  if (!q || !k_codes || !k_meta || !v_codes || !v_meta || !o || !lse)
    return fail(HIFA4_ERR_INVALID_ARGUMENT, "null tensor pointer");
  if ((opt->debug_p_codes == nullptr) != (opt->debug_p_meta == nullptr))
    return fail(HIFA4_ERR_INVALID_ARGUMENT, "debug_p_codes and debug_p_meta must both be set or both be NULL");
  if ((st = check_aligned16({q, k_codes, v_codes, o, s, workspace, opt->debug_p_codes})) != HIFA4_OK) return st;
  if ((st = check_aligned4({k_meta, v_meta, lse, p->cu_seqlens, opt->debug_p_meta})) != HIFA4_OK) return st;
  if (opt->smooth_qk && !s) return fail(HIFA4_ERR_INVALID_ARGUMENT, "smooth_qk set but s is NULL");
  if (d.tokens == 0 || d.S == 0) return HIFA4_OK;
  const size_t need = hifa4_decode_workspace_bytes(p);
  if (!workspace || workspace_bytes < need)
    return fail(HIFA4_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", workspace_bytes, need);
  hipStream_t hs = (hipStream_t)stream;
  hipEvent_t* ev = (hipEvent_t*)opt->timing_events;
  hipError_t e = hipSuccess;
  if (ev && (e = hipEventRecord(ev[0], hs)) != hipSuccess) return hip_fail(e, "timing event");
  hifa4::DecodeLaunch dl;
  dl.q = (const hifa4::half_t*)q;
  dl.s = opt->smooth_qk ? s : nullptr;
  dl.cu = p->cu_seqlens;
  dl.kc = (const uint8_t*)k_codes;
  dl.km = (const uint32_t*)k_meta;
  dl.vc = (const uint8_t*)v_codes;
  dl.vm = (const uint32_t*)v_meta;
  dl.o = (hifa4::half_t*)o;
  dl.lse = lse;
  dl.dbg_codes = (uint8_t*)opt->debug_p_codes;
  dl.dbg_meta = (uint32_t*)opt->debug_p_meta;
  dl.ws = (uint8_t*)workspace;
  dl.ev = ev;
  dl.batch = p->batch;
  dl.S = d.S;
  dl.NB = d.NB;
  dl.hq = p->num_heads_q;
  dl.hkv = p->num_heads_kv;
  dl.D = p->head_dim;
  dl.norm = opt->norm;
  dl.test_no_publish = opt->test_decode_no_publish ? 1 : 0;
  dl.c = (float)(1.4426950408889634 / std::sqrt((double)p->head_dim));
  e = hifa4::launch_decode(dl, hs);
  if (e != hipSuccess) return hip_fail(e, "decode kernels");
  if (ev && (e = hipEventRecord(ev[2], hs)) != hipSuccess) return hip_fail(e, "timing event");
  return HIFA4_OK;
}

hifa4_status hifa4_selftest_exp2(const void* x, void* y, int64_t n, void* stream) {
  if (n < 0 || (n > 0 && (!x || !y))) return fail(HIFA4_ERR_INVALID_ARGUMENT, "bad self-test arguments");
  hipError_t e = hifa4::launch_selftest_exp2((const hifa4::half_t*)x, (hifa4::half_t*)y, (long)n, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "exp2 self-test");
  return HIFA4_OK;
}

hifa4_status hifa4_calibrate_smooth_qk(const hifa4_problem* p, int32_t n_calib, const void* q_calib,
                                       const void* k_calib, float alpha, float* s_out, hifa4_calib_report* report,
                                       void* workspace, size_t workspace_bytes, void* stream) {
  if (!p) return fail(HIFA4_ERR_INVALID_ARGUMENT, "problem is NULL");
  if (n_calib <= 0 || p->max_seqlen <= 0) return fail(HIFA4_ERR_INVALID_ARGUMENT, "n_calib and max_seqlen must be > 0");
  if (p->num_heads_q <= 0 || p->num_heads_kv <= 0 || p->num_heads_q % p->num_heads_kv)
    return fail(HIFA4_ERR_UNSUPPORTED, "num_heads_q must be a positive multiple of num_heads_kv");
  if (p->head_dim != 64 && p->head_dim != 128 && p->head_dim != 256)
    return fail(HIFA4_ERR_UNSUPPORTED, "head_dim %d not in {64, 128, 256}", p->head_dim);
  if (!q_calib || !k_calib || !s_out) return fail(HIFA4_ERR_INVALID_ARGUMENT, "null tensor pointer");
  hifa4_status st = check_aligned16({q_calib, k_calib, workspace});
  if (st == HIFA4_OK) st = check_aligned4({s_out});
  if (st != HIFA4_OK) return st;
  if (!std::isfinite(alpha) || alpha >= 1.0f) return fail(HIFA4_ERR_INVALID_ARGUMENT, "alpha must be finite and < 1");
  const size_t need = hifa4_calibrate_workspace_bytes(p, n_calib);
  if (!workspace || workspace_bytes < need)
    return fail(HIFA4_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", workspace_bytes, need);
  const int hkv = p->num_heads_kv, D = p->head_dim, S = p->max_seqlen;
  const size_t n_stats = (size_t)n_calib * 2 * hkv * D;
  uint32_t* stats = (uint32_t*)workspace;
  unsigned long long* hist = (unsigned long long*)((uint8_t*)workspace + hifa4::round_up256(n_stats * 4));
  hipStream_t hs = (hipStream_t)stream;
  hipError_t e = hifa4::launch_calib((const hifa4::half_t*)q_calib, (const hifa4::half_t*)k_calib, n_calib, S,
                                     p->num_heads_q, hkv, D, stats, hist, hs);
  if (e != hipSuccess) return hip_fail(e, "calibration kernels");
  std::vector<uint32_t> hs_stats(n_stats);
  std::vector<unsigned long long> hh(32768);
  e = hipMemcpyAsync(hs_stats.data(), stats, n_stats * 4, hipMemcpyDeviceToHost, hs);
  if (e == hipSuccess) e = hipMemcpyAsync(hh.data(), hist, 32768 * 8, hipMemcpyDeviceToHost, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  if (e != hipSuccess) return hip_fail(e, "calibration copy-back");

  auto f32 = [](uint32_t u) { float f; std::memcpy(&f, &u, 4); return (double)f; };
  // RMS over calibration sequences of the per-sequence maxima (float64).
  std::vector<double> kbar((size_t)hkv * D), qbar((size_t)hkv * D);
  double kmax_all = 0.0, qmax_all = 0.0;
  for (size_t i = 0; i < (size_t)hkv * D; ++i) {
    double sk = 0.0, sq = 0.0;
    for (int n = 0; n < n_calib; ++n) {
      const double kv = f32(hs_stats[((size_t)n * 2 + 0) * hkv * D + i]);
      const double qv = f32(hs_stats[((size_t)n * 2 + 1) * hkv * D + i]);
      sk += kv * kv;
      sq += qv * qv;
      kmax_all = std::max(kmax_all, kv);
      qmax_all = std::max(qmax_all, qv);
    }
    kbar[i] = std::sqrt(sk / n_calib);
    qbar[i] = std::sqrt(sq / n_calib);
  }
  // P99 of |K| with linear interpolation between order statistics.
  unsigned long long total = 0;
  for (int i = 0; i < 32768; ++i) total += hh[i];
  auto order_stat = [&](unsigned long long k) {
    unsigned long long c = 0;
    for (int i = 0; i < 32768; ++i) {
      c += hh[i];
      if (c > k) {
        const uint16_t bits = (uint16_t)i;
        const _Float16 hv = __builtin_bit_cast(_Float16, bits);
        return (double)(float)hv;
      }
    }
    return 0.0;
  };
  double p99 = 0.0;
  if (total > 0) {
    const double pos = 0.99 * (double)(total - 1);
    const unsigned long long lo = (unsigned long long)std::floor(pos);
    const double t = pos - (double)lo;
    const double a = order_stat(lo), b = order_stat(std::min(lo + 1, total - 1));
    const double diff = b - a;
    p99 = t >= 0.5 ? b - diff * (1.0 - t) : a + diff * t;
  }
  const double rho = p99 > 0 ? kmax_all / p99 : INFINITY;
  const double tkq = qmax_all > 0 ? kmax_all / qmax_all : INFINITY;
  int branch;
  double a_used;
  if (alpha < 0) {
    if (rho >= 6.0 && tkq > 3.0) branch = 2;
    else if (rho >= 6.0 && tkq >= 2.0 && tkq <= 3.0) branch = 1;
    else branch = 0;
    a_used = branch == 2 ? 0.5 : (branch == 1 ? 0.25 : 0.0);
  } else if (alpha == 0) {
    branch = 0;
    a_used = 0.0;
  } else {
    branch = alpha >= 0.5f ? 2 : 1;
    a_used = alpha;
  }
  std::vector<float> sv((size_t)hkv * D, 1.0f);
  if (a_used != 0.0) {
    for (size_t i = 0; i < sv.size(); ++i) {
      const double s = std::pow(kbar[i], a_used) / std::pow(qbar[i], 1.0 - a_used);
      const bool bad = kbar[i] == 0 || qbar[i] == 0 || !std::isfinite(s) || s == 0;
      sv[i] = bad ? 1.0f : (float)s;
    }
  }
  e = hipMemcpyAsync(s_out, sv.data(), sv.size() * 4, hipMemcpyHostToDevice, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  if (e != hipSuccess) return hip_fail(e, "calibration scale upload");
  if (report) {
    report->rho_k = rho;
    report->t_kq = tkq;
    report->branch = branch;
    report->alpha_used = (float)a_used;
  }
  return HIFA4_OK;
}

hifa4_status hifa4_calibrate_smooth_qk_layers(const hifa4_problem* p, int32_t n_layers, int32_t n_calib,
                                              const void* q_calib, const void* k_calib, float alpha, float* s_out,
                                              hifa4_calib_report* reports, void* workspace, size_t workspace_bytes,
                                              void* stream) {
  if (!p) return fail(HIFA4_ERR_INVALID_ARGUMENT, "problem is NULL");
  if (n_layers <= 0) return fail(HIFA4_ERR_INVALID_ARGUMENT, "n_layers must be > 0");
  if (!q_calib || !k_calib || !s_out) return fail(HIFA4_ERR_INVALID_ARGUMENT, "null tensor pointer");
  if (n_calib <= 0 || p->max_seqlen <= 0) return fail(HIFA4_ERR_INVALID_ARGUMENT, "n_calib and max_seqlen must be > 0");
  const size_t q_layer = (size_t)n_calib * p->max_seqlen * p->num_heads_q * p->head_dim;
  const size_t k_layer = (size_t)n_calib * p->max_seqlen * p->num_heads_kv * p->head_dim;
  const size_t s_layer = (size_t)p->num_heads_kv * p->head_dim;
  for (int32_t l = 0; l < n_layers; ++l) {
    const hifa4_status st = hifa4_calibrate_smooth_qk(
        p, n_calib, (const uint16_t*)q_calib + l * q_layer, (const uint16_t*)k_calib + l * k_layer, alpha,
        s_out + l * s_layer, reports ? reports + l : nullptr, workspace, workspace_bytes, stream);
    if (st != HIFA4_OK) {
      const std::string msg = g_last_error;
      return fail(st, "layer %d: %s", l, msg.c_str());
    }
  }
  return HIFA4_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// hifa4_attention_fwd_noalloc: the forward with its K/V pre-pass workspace in
// a file-scope device array (one copy per GPU, held until the process ends),
// for callers that cannot allocate.  In host code `scratch` names a host-side
// stand-in, never the device memory: the device address comes from
// hipGetSymbolAddress, once per device with that device current, and only
// that address is passed to kernels.
static __device__ __align__(256) uint8_t scratch[HIFA4_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

hifa4_status scratch_pointer(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(HIFA4_ERR_UNSUPPORTED, "device index %d above %d", dev, kMaxDevices - 1);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!ptr) return fail(HIFA4_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return HIFA4_OK;
}

}  // namespace

hifa4_status hifa4_attention_fwd_noalloc(const hifa4_problem* p, const hifa4_fwd_options* opt, const void* q,
                                         const void* k, const void* v, const float* s, void* o, float* lse,
                                         void* stream) {
  Dims d;
  hifa4_status st = check_problem(p, &d);
  if (st != HIFA4_OK) return st;
  if (!opt) return fail(HIFA4_ERR_INVALID_ARGUMENT, "options is NULL");
  const size_t need = hifa4_workspace_bytes(p, opt);
  if (need > (size_t)HIFA4_NOALLOC_SCRATCH_BYTES)
    return fail(HIFA4_ERR_WORKSPACE,
                "problem needs %zu bytes of scratch; hifa4_attention_fwd_noalloc holds at most %zu "
                "(use hifa4_attention_fwd with a caller workspace)",
                need, (size_t)HIFA4_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  if ((st = scratch_pointer(&ws)) != HIFA4_OK) return st;
  return hifa4_attention_fwd(p, opt, q, k, v, s, o, lse, ws, (size_t)HIFA4_NOALLOC_SCRATCH_BYTES, stream);
}
