/*
 * hifa4.h -- C ABI of libhifa4: the HiFA4 causal prefill attention forward on
 * AMD Instinct MI355X (gfx950).
 *
 * HiFA4 (arXiv 2607.04302) runs both FlashAttention contractions, QK^T and PV,
 * on 4-bit HIF4 operands while the online-softmax state stays in FP16
 * (Section 3, "C4V16"), with two corrections:
 *   - Smooth-QK (Eq. 1, Sections 4.2-4.4): a calibration-static per-channel
 *     rescale q*s, k/s applied after RoPE, fused into the quantization;
 *   - P-Reordering (Section 4.5, Theorem 1): P is quantized first and the
 *     softmax normalizer is accumulated from that same P^ inside the PV
 *     contraction, through an appended ones block [V^ | 1].
 * Algorithm 1 gives the loop, including the optional Q-Mean auxiliary (the
 * per-token mean of Q~ removed before quantization and added back through the
 * key sums, Section 4.6 and Appendix C).
 *
 * Conventions (all entry points):
 *   - Tensor pointers are DEVICE pointers owned by the caller; the library
 *     never allocates, frees or retains device memory, and keeps no device
 *     state between calls.  Where a host pointer is meant, it says so.
 *   - Alignment: fp16 tensors (q, k, v, o), the scales s, HIF4 code buffers,
 *     workspaces and debug code dumps 16 bytes; metadata buffers, LSE,
 *     cu_seqlens and the calibration output 4 bytes.  Anything else fails with
 *     HIFA4_ERR_INVALID_ARGUMENT before any work is enqueued.
 *   - Fixed-length problems use BSHD layout ([batch, seqlen, heads, dim],
 *     row-major, contiguous).  Variable-length problems pass cu_seqlens and
 *     use THD layout ([total_tokens, heads, dim]).
 *   - fp16 means IEEE binary16, fp32 IEEE binary32.
 *   - Work is enqueued on `stream` (a hipStream_t passed as void*; NULL is the
 *     default stream) and is asynchronous unless stated.  Arguments are
 *     validated synchronously; a launch failure maps to HIFA4_ERR_HIP.
 *     Device faults surface at the caller's next synchronization.
 *   - Nothing throws across the ABI.  On a non-OK status, hifa4_last_error()
 *     returns a message for the calling thread.
 *   - Inputs must be finite and keep |S * log2(e)/sqrt(D)| within the fp16
 *     range (the paper's FP16 softmax state); other inputs are outside the
 *     contract.
 *
 * HIF4 group format (the library's reading; see the HIF4 paragraph of the
 * paper's Background section): 64 elements along the contraction axis of the
 * GEMM that consumes them; an unsigned E6M2 base b (bias 31, byte = e<<2|m,
 * value (1+m/4)*2^(e-31)), the smallest with 1.75*b >= max|x|; level-2 bit j
 * (8 elements) set iff that block's max <= 0.875*b; level-3 bit q (4
 * elements) set iff its max <= 0.875*b*2^-E2[q/2]; a set bit halves the scale;
 * element code u = floor(|x|/step + 1/2) with step = b*2^-(E2+E3)/4, u in 0..7,
 * sign-magnitude nibble sign<<3|u (zero stored as +0).
 *
 * Canonical packed layout, per group: 32 code bytes (element 2i in the low
 * nibble of byte i, element 2i+1 in the high nibble) and one little-endian
 * uint32 of metadata: base | E2 bits << 8 | E3 bits << 16 (bit j = block j).
 * 36 bytes per 64 values = 4.5 bits per value.
 */
#ifndef HIFA4_H
#define HIFA4_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HIFA4_OK = 0,
  HIFA4_ERR_INVALID_ARGUMENT = -1, /* null pointer, bad size or shape        */
  HIFA4_ERR_UNSUPPORTED = -2,      /* valid but not implemented (see below)  */
  HIFA4_ERR_WORKSPACE = -3,        /* workspace too small                    */
  HIFA4_ERR_HIP = -4               /* a HIP runtime call or launch failed    */
} hifa4_status;

/* Shape of one causal prefill problem.  Q has num_heads_q heads, K and V have
 * num_heads_kv; query head h reads key/value head h / (num_heads_q /
 * num_heads_kv) (GQA, Appendix C).  Queries and keys of a sequence have equal
 * lengths and key j is visible to query i iff j <= i.
 *   head_dim     in {64, 128, 256};
 *   max_seqlen   fixed length (BSHD) or, with cu_seqlens, an upper bound of
 *                every sequence length (host value; a longer sequence is
 *                outside the contract: the kernels clamp its length to
 *                max_seqlen, so no access leaves the buffers);
 *   cu_seqlens   NULL for BSHD, else a DEVICE int32 array [batch+1] of
 *                non-decreasing prefix sums starting at 0 (THD layout);
 *   total_tokens with cu_seqlens: cu_seqlens[batch] (host value); ignored
 *                for BSHD (batch*max_seqlen);
 *   causal       must be 1. */
typedef struct {
  int32_t batch;
  int32_t num_heads_q;
  int32_t num_heads_kv;
  int32_t head_dim;
  int32_t max_seqlen;
  const int32_t* cu_seqlens;
  int32_t total_tokens;
  int32_t causal;
} hifa4_problem;

typedef enum {
  HIFA4_NORM_PREORDER = 0,     /* P-Reordering: l accumulates P^ (Section 4.5) */
  HIFA4_NORM_INCONSISTENT = 1  /* Direct baseline: l accumulates pre-quantization
                                  P while PV uses P^ (Theorem 1, "mismatched") */
} hifa4_norm;

typedef enum {
  HIFA4_OPERANDS_HIF4 = 0,   /* both contractions on HIF4 operands (C4V16)     */
  HIFA4_OPERANDS_FP16 = 1,   /* same loop on fp16 operands, no quantization and
                                no smoothing: the FP16 reference (C16V16) */
  HIFA4_OPERANDS_P_ONLY = 2  /* P-only local operator (the study the paper
                                defers, Section 4.5): Q, K and V stay fp16
                                (no smoothing), scores and softmax as in the
                                FP16 reference, P^ = HIF4(P) feeds the PV
                                product; the normalizer follows opt->norm */
} hifa4_operands;

/* Options of hifa4_attention_fwd.
 *   smooth_qk      0: the scale vector is ignored (treated as all ones);
 *   debug_p_codes  NULL, or a DEVICE uint8 buffer [NH, NT, NB, 32]
 *                  receiving the canonical codes of the P^ groups of query
 *                  heads [h0, h0+NH) and tokens [t0, t0+NT) (the dump window,
 *                  below), NB = ceil(max_seqlen/64); entry (h-h0, t-t0, J) is
 *                  written for the 64-key blocks J <= i/64 that query t
 *                  (position i in its sequence) sees, other entries are left
 *                  untouched;
 *   debug_p_meta   NULL, or a DEVICE uint32 buffer [NH, NT, NB] with the
 *                  matching metadata words.  Both or neither.
 *   debug_head_begin/_count, debug_token_begin/_count  the dump window
 *                  h0, NH, t0, NT; a count of 0 means every query head
 *                  (every token, T = batch*max_seqlen for BSHD) and needs a
 *                  begin of 0; a window outside the problem fails with
 *                  HIFA4_ERR_INVALID_ARGUMENT.
 * Debug dumps are produced for HIFA4_OPERANDS_HIF4 and _P_ONLY.
 *   timing_events  NULL, or a HOST array of three hipEvent_t (created by the
 *                  caller) that the call records on `stream` before the K/V
 *                  pre-pass, between the pre-pass and the attention kernel,
 *                  and after the attention kernel -- per-kernel device time
 *                  without a profiler.  The events are not waited on.
 *   q_mean         0 or 1: the Q-Mean auxiliary (Algorithm 1; Section 4.6;
 *                  Appendix C).  Per query row mu = fp16(exact sum of the
 *                  row's D smoothed values / D); the row is quantized as
 *                  Q_z = fp16(q~ - mu); per key kappa = fp32(exact sum of the
 *                  key's smoothed channels); after the group terms the score
 *                  accumulator takes fp32(S_acc + mu*kappa) (the exact
 *                  product added with one rounding), before the multiply by
 *                  c.  HIF4 operands only (HIFA4_ERR_UNSUPPORTED with FP16
 *                  operands).
 *   test_decode_no_publish  testing only; see hifa4_decode_fwd (0 otherwise). */
typedef struct {
  int32_t norm;       /* hifa4_norm      */
  int32_t operands;   /* hifa4_operands  */
  int32_t smooth_qk;
  void* debug_p_codes;
  void* debug_p_meta;
  void** timing_events;
  int32_t q_mean;
  int32_t test_decode_no_publish;  /* testing only, hifa4_decode_fwd: see there */
  int32_t debug_head_begin;        /* P^ dump window of hifa4_attention_fwd */
  int32_t debug_head_count;
  int32_t debug_token_begin;
  int32_t debug_token_count;
} hifa4_fwd_options;

/* Host-side calibration report (Table 1 statistics and the gate decision). */
typedef struct {
  double rho_k;        /* max|K| / P99(|K|) over all calibration K elements */
  double t_kq;         /* max|K| / max|Q|                                     */
  int32_t branch;      /* 0 bypass, 1 mild, 2 strong                          */
  float alpha_used;
} hifa4_calib_report;

/* Bytes of device workspace hifa4_attention_fwd needs for this problem and
 * options (0 on invalid arguments).  The workspace holds the MFMA-ready K and
 * V operands written by the pre-pass. */
size_t hifa4_workspace_bytes(const hifa4_problem* p, const hifa4_fwd_options* opt);

/* Bytes of device workspace hifa4_calibrate_smooth_qk needs. */
size_t hifa4_calibrate_workspace_bytes(const hifa4_problem* p, int32_t n_calib);

/* Offline Smooth-QK calibration (Eq. 1; Sections 4.3-4.4; Appendix C).
 * q_calib: DEVICE fp16 [n_calib, max_seqlen, num_heads_q, head_dim];
 * k_calib: DEVICE fp16 [n_calib, max_seqlen, num_heads_kv, head_dim]
 * (n_calib fixed-length sequences stacked on the leading axis; p->batch and
 * p->cu_seqlens are ignored).  Per sequence, the GPU reduces max|K| over
 * tokens and max|Q| over tokens and the query heads of each group, per (kv
 * head, channel), and a 32768-bin histogram of |K| (exact for fp16).  On the
 * host, in float64: the RMS over sequences, s = Kbar^alpha / Qbar^(1-alpha)
 * rounded once to fp32 (s = 1 where a statistic is 0 or s is not finite),
 * and the gate statistics rho_K = max|K| / P99|K| (linear interpolation
 * between order statistics) and T = max|K| / max|Q|.
 *   alpha > 0  use this alpha;  alpha == 0  bypass (s = 1);
 *   alpha < 0  the gate picks: strong (0.5) if rho_K >= 6 and T > 3,
 *              mild (0.25) if rho_K >= 6 and 2 <= T <= 3, else bypass.
 * s_out: DEVICE fp32 [num_heads_kv, head_dim].  report: HOST, may be NULL.
 * workspace: DEVICE, at least hifa4_calibrate_workspace_bytes().
 * Synchronizes `stream` before returning (an offline call). */
hifa4_status hifa4_calibrate_smooth_qk(const hifa4_problem* p, int32_t n_calib,
                                       const void* q_calib, const void* k_calib,
                                       float alpha, float* s_out,
                                       hifa4_calib_report* report,
                                       void* workspace, size_t workspace_bytes,
                                       void* stream);

/* Offline calibration of several layers in one call (Sections 4.3-4.4 and
 * Appendix F: the statistics, the scale and the gate decision are taken per
 * layer).  Layer l reads q_calib + l * (n_calib*max_seqlen*num_heads_q*head_dim)
 * and k_calib + l * (n_calib*max_seqlen*num_heads_kv*head_dim) fp16 elements
 * (DEVICE, layers stacked on a leading axis) and writes s_out + l*num_heads_kv*
 * head_dim (DEVICE fp32) and reports[l] (HOST, may be NULL); each layer is
 * exactly hifa4_calibrate_smooth_qk on its slice, with the same alpha (alpha < 0
 * lets the gate decide per layer).  workspace: DEVICE, at least
 * hifa4_calibrate_workspace_bytes(p, n_calib), reused by every layer.
 * Synchronizes `stream`.  On an error no later layer is processed. */
hifa4_status hifa4_calibrate_smooth_qk_layers(const hifa4_problem* p, int32_t n_layers,
                                              int32_t n_calib, const void* q_calib,
                                              const void* k_calib, float alpha, float* s_out,
                                              hifa4_calib_report* reports, void* workspace,
                                              size_t workspace_bytes, void* stream);

/* Smooth-QK then HIF4 quantization of Q~ = fp16(q*s) and K~ = fp16(k/s),
 * each the exact product or quotient of the fp16 input and the fp32 scale
 * rounded once to fp16 (nearest even), in groups of 64 consecutive channels
 * of each (token, head) row (Algorithm 1, the Smooth-QK and HIF4 steps).
 * q, k: DEVICE fp16 in the problem's layout; s: DEVICE fp32
 * [num_heads_kv, head_dim] or NULL (no smoothing).
 * Outputs (DEVICE, canonical layout):
 *   q_codes uint8 [T, num_heads_q, head_dim/64, 32], q_meta uint32 [T, Hq, D/64]
 *   k_codes uint8 [T, num_heads_kv, head_dim/64, 32], k_meta uint32 [T, Hkv, D/64]
 * where T is the token count.  q, q_codes and q_meta may all be NULL: then
 * only K^ is written (filling or appending to a K^ cache; rows are
 * independent, so the K^ of new tokens can be written in place at their
 * cache rows).  Asynchronous. */
hifa4_status hifa4_quantize_qk(const hifa4_problem* p, const void* q, const void* k,
                               const float* s, void* q_codes, void* q_meta,
                               void* k_codes, void* k_meta, void* stream);

/* HIF4 quantization of V along tokens (the contraction axis of PV): groups
 * of 64 consecutive tokens of one (kv head, channel) column, aligned to each
 * sequence's first token; a partial last group is zero padded.
 * v: DEVICE fp16 in the problem's layout.  Outputs (DEVICE, canonical):
 *   v_codes uint8 [batch, NB, num_heads_kv, head_dim, 32]
 *   v_meta  uint32 [batch, NB, num_heads_kv, head_dim]
 * with NB = ceil(max_seqlen/64); groups past a sequence's end are written as
 * all-zero groups.  Asynchronous. */
hifa4_status hifa4_quantize_v(const hifa4_problem* p, const void* v, void* v_codes,
                              void* v_meta, void* stream);

/* The HiFA4 causal prefill forward (Algorithm 1; Section 4.5).
 * q: DEVICE fp16 [.., num_heads_q, head_dim]; k, v: DEVICE fp16
 * [.., num_heads_kv, head_dim]; s: DEVICE fp32 [num_heads_kv, head_dim] (may be
 * NULL when opt->smooth_qk == 0 or operands are FP16).
 * Per query row and 64-key block in ascending order, with c =
 * fp32(log2(e)/sqrt(D)): per 64-channel group g the exact term t_g = the dot
 * of the dequantized Q^ and K^ groups; S_acc = the fp32 sum of the t_g in
 * group order, each addition rounded once (with Q-Mean, then
 * fp32(S_acc + mu*kappa)); S2 = fp16(fp32(S_acc * c));
 * m_new = max(m, rowmax S2); P = fp16(2^(S2-m_new));
 * r = fp16(2^(m-m_new)); P^ = HIF4(P); O = r*O + P^ V^ and l = r*l + P^ 1
 * (fp32 accumulation); O_out = fp16(O/l), LSE = m*ln2 + ln(l).
 * o: DEVICE fp16, same layout as q.  lse: DEVICE fp32 [num_heads_q, T] (T the
 * token count, natural log of the softmax partition, including the score
 * scale 1/sqrt(D)).  workspace: DEVICE, >= hifa4_workspace_bytes().
 * Asynchronous. */
hifa4_status hifa4_attention_fwd(const hifa4_problem* p, const hifa4_fwd_options* opt,
                                 const void* q, const void* k, const void* v,
                                 const float* s, void* o, float* lse,
                                 void* workspace, size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops, harnesses that forbid hipMalloc): hifa4_attention_fwd
 * with its workspace in a static device array of the library,
 * HIFA4_NOALLOC_SCRATCH_BYTES (32 MiB) per GPU, held from the first call on
 * that GPU until the process ends.  The caller passes inputs and outputs as
 * for hifa4_attention_fwd; the call allocates and frees nothing.  A problem
 * whose hifa4_workspace_bytes() exceeds the array fails with
 * HIFA4_ERR_WORKSPACE before any work is enqueued (32 MiB holds, for
 * example, 8 kv heads of D=128 up to 10240 tokens).  The array's address on
 * the current device (which must be the stream's device) is looked up on the
 * first call there.  Every call on one GPU shares its array: calls that
 * overlap on one GPU (different streams, or threads) race and give wrong
 * results; calls ordered on one stream are safe.  Nothing in the array needs
 * to start at zero (each call writes every entry it reads).  Otherwise
 * identical to hifa4_attention_fwd, including the debug and timing options. */
#define HIFA4_NOALLOC_SCRATCH_BYTES (32u << 20)
hifa4_status hifa4_attention_fwd_noalloc(const hifa4_problem* p, const hifa4_fwd_options* opt,
                                         const void* q, const void* k, const void* v,
                                         const float* s, void* o, float* lse, void* stream);

/* Workspace size in bytes of hifa4_decode_fwd for problem p (0 if p is
 * invalid).  It grows with batch * num_heads_q * ceil(max_seqlen/64). */
size_t hifa4_decode_workspace_bytes(const hifa4_problem* p);

/* One decode step of HiFA4 over a packed HIF4 K/V cache: for each sequence b,
 * the attention of its newest token (position L_b - 1, which sees every cached
 * key) -- row L_b - 1 of hifa4_attention_fwd on the same sequence, computed
 * from the cache.  The paper evaluates prefill only and leaves decode and
 * the KV-cache footprint open; this entry point applies Algorithm 1 and
 * Section 4.5 to that row with the same contract, including every P^ code.
 * p describes the cached sequences (their lengths include the newest token):
 * BSHD (every length max_seqlen) or THD with cu_seqlens; causal must be 1.
 * q: DEVICE fp16 [batch, num_heads_q, head_dim], the raw query of each
 *    sequence's newest token (smoothed here with s when opt->smooth_qk);
 * k_codes/k_meta: DEVICE canonical K^ cache [T, Hkv, D/64, 32] / [T, Hkv, D/64]
 *    as written by hifa4_quantize_qk with the same s (T the token count);
 * v_codes/v_meta: DEVICE canonical V^ cache [batch, NB, Hkv, D, 32] /
 *    [batch, NB, Hkv, D] as written by hifa4_quantize_v (NB = ceil(max_seqlen/64));
 * o: DEVICE fp16 [batch, num_heads_q, head_dim]; lse: DEVICE fp32
 *    [num_heads_q, batch]; rows of empty sequences are left untouched.
 * opt: norm, smooth_qk, debug_p_codes/_meta ([num_heads_q, batch, NB, 32] /
 *    [num_heads_q, batch, NB], entries J < ceil(L_b/64) written) and
 *    timing_events (before the first kernel, before the merge kernel, after
 *    the merge) as for hifa4_attention_fwd; operands must be
 *    HIFA4_OPERANDS_HIF4 and q_mean 0 (the cache carries no key sums), else
 *    HIFA4_ERR_UNSUPPORTED; num_heads_q / num_heads_kv must be <= 8 (else
 *    HIFA4_ERR_UNSUPPORTED).
 * workspace: DEVICE, >= hifa4_decode_workspace_bytes(p).  Asynchronous.
 * Where the splits of the key range fill the GPU (at least 256 workgroups),
 * scores and splits run in one kernel in which each split waits, with a
 * bounded spin, for the run maxima that the splits before it in the same row
 * publish (tagged with a per-call value; the last kernel of the call clears
 * them, so no word of an earlier call, eager or replayed from a graph,
 * satisfies a wait).  The waits end because every GPU engine dispatches the
 * workgroups of a grid in index order and each waits only on lower indices;
 * if a wait nevertheless gives up, that row's o and lse are NaN (never a
 * silently wrong value).  opt->test_decode_no_publish != 0 (testing only)
 * publishes nothing and lets every wait give up after 16 polls, so that the
 * rows of every split after the first come out NaN. */
hifa4_status hifa4_decode_fwd(const hifa4_problem* p, const hifa4_fwd_options* opt,
                              const void* q, const void* k_codes, const void* k_meta,
                              const void* v_codes, const void* v_meta, const float* s,
                              void* o, float* lse, void* workspace, size_t workspace_bytes,
                              void* stream);

/* Device self-test of the kernels' fp16 exponential: y[i] = fp16(2^x[i]) for
 * n fp16 inputs x (DEVICE, fp16 bits), evaluated by the same device routine
 * the attention kernel uses.  Asynchronous. */
hifa4_status hifa4_selftest_exp2(const void* x, void* y, int64_t n, void* stream);

/* Message for the last non-OK status returned on the calling thread. */
const char* hifa4_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* HIFA4_H */
