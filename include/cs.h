/*
 * cs.h -- C ABI of the MI355X (gfx950) cached N-candidate DiT rollout.
 *
 * The library runs CachedSearch's exploration loop (Alg. 1 of the paper):
 * N candidate latents, one per seed, are integrated through T Euler steps of
 * the flow-matching ODE (Sec. Preliminaries, Eq. euler) with optional
 * classifier-free guidance (Eq. cfg).  At every step and for every candidate
 * and guidance branch, the transformation-vector cache (Sec. Adaptive
 * transformation-vector caching, Eqs. delta, skip, indicator) decides whether
 * the transformer is evaluated or its cached residual reused.  The final
 * latents are scored and ranked; the ranking is compared with the full
 * (uncached) rollouts of the same seeds by Spearman correlation (Sec.
 * Experiments, definitions and protocol).
 *
 * Conventions
 *  - Pointers documented "device" are HIP device pointers; "host" pointers
 *    are ordinary CPU memory.  The caller owns every pointer it passes.
 *  - cs_model_init copies the weights into memory the model owns; the
 *    caller's weight buffer may be freed after the call returns.  A rollout
 *    owns its state and workspace and frees them in cs_rollout_free.
 *  - All device work is enqueued on the HIP stream given at init (void* is a
 *    hipStream_t; NULL = the default stream).  Calls that write host outputs
 *    synchronise that stream before returning.
 *  - Every function returns a cs_status; no exception or abort crosses the
 *    ABI.  On failure, cs_last_error() returns a message (thread-local).
 *    Arguments are validated before any device work is enqueued, so a
 *    CS_E_INVAL/CS_E_STATE return leaves the device untouched.
 *  - Identical inputs give bitwise identical outputs, independent of N and
 *    of which other candidates are evaluated in the same step (no atomics,
 *    fixed reduction orders, tile shapes fixed per model).
 *  - Latents are float32 [C][F][H][W] per candidate, candidates contiguous.
 *    D = C*F*H*W.  Weights: see cs_model_weight_count.
 */
#ifndef CACHEDSEARCH_CS_H
#define CACHEDSEARCH_CS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CS_OK = 0,
  CS_E_INVAL = 1,        /* bad argument (null, out of range, NaN, shape)  */
  CS_E_NOMEM = 2,        /* device or host allocation failed               */
  CS_E_DEVICE = 3,       /* a HIP call failed (message names it)           */
  CS_E_STATE = 4,        /* call out of order (e.g. step k+2 after k)      */
  CS_E_UNSUPPORTED = 5   /* valid but not supported shape/config           */
} cs_status;

typedef enum { CS_BF16 = 0, CS_FP32 = 1 } cs_dtype;

/* Cache modes.  OFF computes every call (recovers the uncached rollout
 * G(c,s)); ADAPTIVE applies the accumulated drift rule with threshold tau;
 * STATIC computes every static_k-th step between warmup and cooldown (the
 * uniform-schedule baseline of Sec. Method, properties paragraph).
 * PAB is attention-output broadcasting, one of the published engines the
 * paper compares (Sec. Ranking preservation across published caching
 * methods, Table tab:baselines): every call runs the transformer, but each
 * block's self- and cross-attention output (after the output projection,
 * before the self-attention gate) is recomputed only every
 * pab_self_range / pab_cross_range steps and reused in between.  Steps
 * 1..k_warm and n_steps-k_cool+1..n_steps recompute both; a step s in
 * between recomputes a branch of range r iff (s - k_warm) % r == 0 or
 * nothing is stored yet.  PAB keeps two [n_blocks][N*B][tokens][hidden]
 * arrays of the compute type on the device. */
typedef enum {
  CS_CACHE_OFF = 0, CS_CACHE_ADAPTIVE = 1, CS_CACHE_STATIC = 2, CS_CACHE_PAB = 3
} cs_cache_mode;

/* Transformer shape.  The paper treats the velocity model v_theta(x, t, c)
 * as a black box (Sec. Preliminaries); the library implements a Wan-shaped
 * DiT: 1x2x2 patch embedding, n_blocks of [adaLN self-attention with
 * RMSNorm q/k and 3D RoPE, cross-attention to the text embedding,
 * adaLN tanh-GELU FFN], adaLN head.  Requirements: hidden = heads*head_dim,
 * head_dim in {32, 64, 128}, hidden % 64 == 0, ffn % 64 == 0,
 * text_dim % 64 == 0, in_ch % 16 == 0, freq_dim == 256, patch = (1,2,2),
 * lat_h and lat_w even.  dtype selects the transformer's matrix arithmetic (bf16 operands
 * with fp32 accumulation, or fp32 throughout); the cache state, latents,
 * residual stream and all reductions are fp32/fp64 in both modes. */
typedef struct {
  int32_t n_blocks, hidden, heads, head_dim, ffn;
  int32_t text_dim, text_len, freq_dim;
  int32_t in_ch, lat_f, lat_h, lat_w;
  int32_t patch_t, patch_h, patch_w;
  int32_t dtype;                 /* cs_dtype */
} cs_model_desc;

/* Rollout description (Alg. 1 inputs: seeds via x1, tau, mode).
 * n_branch: 1 = conditional only, 2 = CFG with guidance scale `guidance`
 * (branch 0 conditional, branch 1 unconditional).  Steps are 1-based; steps
 * 1..k_warm and n_steps-k_cool+1..n_steps always compute, as does any call
 * before the branch's first Delta exists.  tau >= 0, +INF allowed.
 * timesteps: host, n_steps+1 floats, timesteps[0] = 1 > ... >
 * timesteps[n_steps] = 0, strictly decreasing (copied at init). */
typedef struct {
  int32_t n_cand, n_steps, n_branch, k_warm, k_cool, static_k;
  int32_t mode;                  /* cs_cache_mode */
  float tau, guidance;
  const float* timesteps;
  int32_t pab_self_range;        /* >= 1, read in CS_CACHE_PAB mode only  */
  int32_t pab_cross_range;       /* >= 1, read in CS_CACHE_PAB mode only  */
} cs_rollout_desc;

typedef struct cs_model cs_model;
typedef struct cs_rollout cs_rollout;

/* Per-rollout counters, read by cs_rollout_stats. */
typedef struct {
  int32_t steps_done;            /* last completed step (0 after init)     */
  int64_t calls;                 /* transformer calls requested (N*B*steps)*/
  int64_t computed;              /* calls evaluated by the transformer     */
  int64_t self_reused;           /* PAB: calls that reused the stored      */
  int64_t cross_reused;          /*   self / cross attention outputs       */
  int32_t n_cand;                /* current candidate count (after retain) */
} cs_rollout_stats_t;

/* Kernel families timed by the optional profiler (cs_profile_*). */
typedef enum {
  CS_K_SELF_ATTN = 0, CS_K_CROSS_ATTN = 1, CS_K_GEMM = 2, CS_K_NORM = 3,
  CS_K_DECIDE = 4, CS_K_UPDATE = 5, CS_K_SCORE = 6, CS_K_OTHER = 7,
  CS_K_COUNT = 8
} cs_kernel_family;

/* ---------------------------------------------------------------- model */

/* Number of float32 values in the flat weight array for `desc`.  Order:
 * patch_w[d][p] patch_b[d] text1_w[d][text_dim] text1_b[d] text2_w[d][d]
 * text2_b[d] time1_w[d][256] time1_b[d] time2_w[d][d] time2_b[d]
 * mod_w[6d][d] mod_b[6d], then per block: mod[6][d] (shift1, scale1,
 * gate1, shift2, scale2, gate2) qkv_w[3d][d] qkv_b[3d] q_gain[d] k_gain[d]
 * o_w[d][d] o_b[d] ca_ln_g[d] ca_ln_b[d] caq_w caq_b cak_w cak_b cav_w
 * cav_b ([d][d], [d]) caq_gain[d] cak_gain[d] cao_w[d][d] cao_b[d]
 * ffn1_w[ffn][d] ffn1_b[ffn] ffn2_w[d][ffn] ffn2_b[d], then head_mod[2][d]
 * (shift, scale) head_w[p][d] head_b[p], with d = hidden and
 * p = in_ch*patch_t*patch_h*patch_w.  Matrices are [out][in] row-major. */
cs_status cs_model_weight_count(const cs_model_desc* desc, size_t* count);

/* Build a model.  weights: device, float32, cs_model_weight_count values
 * (copied; matrices rounded to bf16 round-to-nearest-even in CS_BF16 mode,
 * vectors kept fp32).  stream: hipStream_t or NULL.  On success *out owns
 * device memory until cs_model_free. */
cs_status cs_model_init(const cs_model_desc* desc, const float* weights, size_t n_weights,
                        void* stream, cs_model** out);
void cs_model_free(cs_model* model);

/* One transformer evaluation v_theta(x, t, c) (Sec. Preliminaries) for n
 * latents sharing the timestep t and one text context.  x: device
 * [n][D] float32; ctx: device [text_len][text_dim] float32; v: device
 * [n][D] float32 (may not alias x).  Enqueued on the model's stream. */
cs_status cs_velocity(cs_model* model, const float* x, int32_t n, float t, const float* ctx,
                      float* v);

/* -------------------------------------------------------------- rollout */

/* Start a generation (Alg. 1: reset cache state, then G_tau(c, s_i) for
 * every seed).  x1: device [n_cand][D] float32 initial noise (copied).
 * ctx_cond / ctx_uncond: device [text_len][text_dim] float32; ctx_uncond
 * must be non-NULL iff n_branch == 2 (copied into per-branch cross-attention
 * keys/values here, once per rollout).  All cache state is zeroed.  In
 * CS_CACHE_PAB mode both ranges must be >= 1 (else CS_E_INVAL) and the two
 * attention-output arrays are allocated here (CS_E_NOMEM if they do not
 * fit). */
cs_status cs_rollout_init(cs_model* model, const cs_rollout_desc* desc, const float* x1,
                          const float* ctx_cond, const float* ctx_uncond, cs_rollout** out);
void cs_rollout_free(cs_rollout* r);

/* Cache decision for step `step` (must be the next step, 1..n_steps) for
 * every candidate i and branch b (Eq. indicator and its rule): forced
 * calls compute; otherwise a_ib += ||x_i - xref_ib||_F / ||xref_ib||_F and
 * the call is skipped iff a_ib <= tau (a call with ||xref|| = 0 computes).
 * override_mask: NULL, or host [n_cand][n_branch] bytes (1 = compute) that
 * replace the rule's decisions (replay); the indicator is still accumulated
 * and reported.  An override that skips a call with no cached residual (in
 * CS_CACHE_OFF mode, or before that branch's first computed call) is
 * rejected with CS_E_INVAL before any device work.  mask_out: NULL or host [n_cand][n_branch] (1 = compute).
 * a_out: NULL or host [n_cand][n_branch], the indicator value compared with
 * tau at this step, NaN where the call was forced.  Calling it twice for
 * the same step returns CS_E_STATE.  In CS_CACHE_PAB mode every call
 * computes (mask all 1, a NaN) unless overridden. */
cs_status cs_cache_decide(cs_rollout* r, int32_t step, const uint8_t* override_mask,
                          uint8_t* mask_out, double* a_out);

/* Execute step `step`: evaluate the transformer for the computed calls,
 * refresh Delta = v - x and x_ref = x on them (Eq. delta), form x + Delta on
 * the skipped ones (Eq. skip), combine branches (Eq. cfg) and take the
 * Euler step (Eq. euler).  Runs cs_cache_decide(step, NULL, NULL, NULL)
 * first if it was not called for this step.  In CS_CACHE_PAB mode the
 * attention outputs follow the broadcast schedule described with
 * cs_cache_mode; a replay override is then not allowed (CS_E_UNSUPPORTED
 * from cs_cache_decide). */
cs_status cs_denoise_step(cs_rollout* r, int32_t step);

/* Scores s_i = <w, x_i> / sqrt(D) of the current latents, summed in fp64 in
 * a fixed order (the stand-in verifier of Alg. 1).  w: device [D] float32;
 * scores: host [n_cand] double.  Synchronises. */
cs_status cs_score(cs_rollout* r, const float* w, double* scores);

/* Allocation-free scoring, for callers that cannot allocate device memory
 * (code under HIP graph capture, serving loops or harnesses that forbid
 * hipMalloc): the scores of cs_score, s_i = <w, x_i> / sqrt(D) summed in
 * fp64 in the same fixed order (bitwise equal to cs_score on the same
 * latents), for n latents the caller holds, without a rollout handle.
 * x: device [n][D] float32, w: device [D] float32, both 16-byte aligned;
 * D % 4 == 0; scores: device [n] double (written); stream: hipStream_t or
 * NULL.  Only enqueues work (no synchronisation, no allocation, no memset).
 * The per-chunk partial sums go to a static device array owned by the
 * library, CS_SCORE_NOALLOC_MAX_PARTIALS doubles (4 MiB) per GPU, held until
 * the process ends; n * ceil(D / 8192) above that capacity returns
 * CS_E_INVAL before any device work.  Every call on one GPU shares that
 * array and it keeps the last call's contents: calls that overlap on one
 * GPU (different streams, or host threads) race and must be serialised by
 * the caller. */
#define CS_SCORE_NOALLOC_MAX_PARTIALS (512 * 1024)
cs_status cs_score_noalloc(const float* x, const float* w, int32_t n, int64_t D, double* scores,
                           void* stream);

/* Pruned composition (Sec. Composition with pruned search).
 * cs_rollout_enable_preview(r, 1) makes every following cs_denoise_step also
 * keep the guided velocity v~ of that step (one extra [n_cand][D] fp32
 * buffer, allocated here; 0 frees it).  cs_preview_score then scores the
 * sampler's x0 estimate after the last completed step k,
 * x0_hat = x_{t_{k+1}} - t_{k+1} v~_k, as <w, x0_hat>/sqrt(D) (fp64, fixed
 * order); it returns CS_E_STATE unless the preview was enabled before step
 * k.  w: device [D]; scores: host [n_cand].  Synchronises.
 * cs_rollout_retain keeps only the candidates keep[0..n_keep-1] (host,
 * strictly increasing indices in the current numbering) with their complete
 * cache state; they are renumbered 0..n_keep-1 and n_cand becomes n_keep.
 * Not allowed between cs_cache_decide and cs_denoise_step (CS_E_STATE),
 * nor in CS_CACHE_PAB mode (CS_E_UNSUPPORTED).  Synchronises. */
cs_status cs_rollout_enable_preview(cs_rollout* r, int32_t on);
cs_status cs_preview_score(cs_rollout* r, const float* w, double* scores);
cs_status cs_rollout_retain(cs_rollout* r, const int32_t* keep, int32_t n_keep);

/* Copy the current latents to dst: device [n_cand][D] float32. */
cs_status cs_rollout_latents(cs_rollout* r, float* dst);

cs_status cs_rollout_stats(cs_rollout* r, cs_rollout_stats_t* out);

/* Checkpoint: the complete rollout state {step, x, x_ref, Delta, a,
 * has_ref}.  cs_rollout_export with buf == NULL stores the required size in
 * *bytes; otherwise buf (host) must hold *bytes bytes.  cs_rollout_import
 * restores a state exported from a rollout with the same model and
 * description.  Both synchronise.  Not available in CS_CACHE_PAB mode,
 * whose state includes the attention-output arrays (CS_E_UNSUPPORTED). */
cs_status cs_rollout_export(cs_rollout* r, void* buf, size_t* bytes);
cs_status cs_rollout_import(cs_rollout* r, const void* buf, size_t bytes);

/* ---------------------------------------------------------------- ranking */

/* Host only, thread-safe.  Orders candidates by decreasing score (equal
 * scores: lower index first) for both score vectors, and computes the
 * Spearman correlation of average ranks (NaN if a vector is constant) and
 * top-1 agreement (Sec. Experiments, definitions and protocol; Alg. 1's
 * argmax).  s_cached, s_full: host [n] doubles; order_cached, order_full:
 * host [n] int32 (position 0 = best).  n >= 2 else CS_E_INVAL; scores must
 * not be NaN.  Any output pointer may be NULL.
 * Order only: with s_full == NULL only order_cached is written (n >= 1);
 * order_full, rho and top1_agree must then be NULL (else CS_E_INVAL).  This
 * is the ranking step of a search without a reference: keep mode's argmax
 * (order_cached[0]) and the top-k of pruned search. */
cs_status cs_rank(const double* s_cached, const double* s_full, int32_t n, int32_t* order_cached,
                  int32_t* order_full, double* rho, int32_t* top1_agree);

/* ---------------------------------------------------------------- profiler */

/* Enable (1) or disable (0) HIP-event timing of every kernel launch the
 * rollout (and its model's cs_velocity) enqueues, per cs_kernel_family.
 * cs_profile_read synchronises, then reports the summed device time in ms
 * and the number of launches since the last reset. */
cs_status cs_profile_enable(cs_model* model, int32_t on);
cs_status cs_profile_reset(cs_model* model);
cs_status cs_profile_read(cs_model* model, int32_t family, double* total_ms, int64_t* launches);

/* Thread-local description of the last failure in this thread. */
const char* cs_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* CACHEDSEARCH_CS_H */
