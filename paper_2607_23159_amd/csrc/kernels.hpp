// Launchers of the gfx950 kernels.  All take a HIP stream and return the
// launch status; shapes are validated by the runtime before any launch.
#pragma once
#include "common.hpp"

namespace cs {

// ---- GEMM (k_gemm.hip).  W is [N][K] (K contiguous); every variant adds a
// bias vector (non-NULL) in its epilogue.  bf16 weights are stored in the
// tiled layout of gemm_tile_weight, fp32 weights row-major.
long gemm_tiled_weight_elems(int N, int K);
hipError_t gemm_tile_weight(const float* src, int N, int K, bf16* dst, hipStream_t st);
template <typename T>
hipError_t gemm_store(const T* A, long lda, const T* W, int M, int N, int K, const float* bias,
                      int act, T* out, long ldo, hipStream_t st);
template <typename T>
hipError_t gemm_store_t(const T* A, long lda, const T* W, int M, int N, int K, const float* bias,
                        T* out, long ldo, hipStream_t st);
template <typename T>
hipError_t gemm_qkv(const T* A, const T* W, int M, int d, const float* bias, int L, T* qk, T* vt,
                    long vt_ld, hipStream_t st);
// z[M][N] += gate * (A W^T + bias) (gate NULL: 1); when y is non-NULL the
// branch output A W^T + bias is also stored to y[M][N] in the compute type.
template <typename T>
hipError_t gemm_residual(const T* A, long lda, const T* W, int M, int N, int K, const float* bias,
                         const float* gate, float* z, T* y, hipStream_t st);
template <typename T>
hipError_t gemm_patch(const T* A, const T* W, int M, int d, int P, const float* bias, float* z,
                      hipStream_t st);
template <typename T>
hipError_t gemm_head(const T* A, const T* W, int M, int d, int P, const float* bias, float* out,
                     const int* slot_id, int L, int gh, int gw, int F, int H, int Wd, long D,
                     hipStream_t st);

// ---- attention (k_attn.hip)
template <typename T> struct AttnArgs {
  const T* q; long q_ld; long q_ss;     // stream s: rows at q + s*q_ss, row stride q_ld
  const T* k; long k_ld; long k_ss;     // keys of kv stream j at k + j*k_ss
  const T* vt; long vt_ld; long vt_ss;  // values transposed: row = channel, col = key
  const int* kv_sel;                    // stream -> kv stream (NULL: identity, self-attention)
  T* o; long o_ld; long o_ss;
  int lq, lk, heads, n_streams;
  float scale_log2;                     // log2(e) / sqrt(head_dim)
};
// Required padding of the key dimension of vt (columns), and of k rows.
int attn_kv_tile(int dtype_bytes, int head_dim);
template <typename T> hipError_t flash_attention(const AttnArgs<T>& a, int head_dim, hipStream_t st);

// ---- row kernels (k_rows.hip)
// u = LN(z) * (1 + scale) + shift   (mode 0, shift/scale vectors)
// u = LN(z) * gain + bias           (mode 1)
template <typename T>
hipError_t layer_norm_mod(const float* z, long rows, int d, const float* shift_or_gain,
                          const float* scale_or_bias, int mode, T* u, hipStream_t st);
// In-place RMSNorm (gain) over the first d columns of each row of x (row
// stride ld, `parts` consecutive d-wide parts per row, each its own norm),
// then optional 3D RoPE per head with table rope[token][head_dim/2]
// (cos, sin), token = row % L.
template <typename T>
hipError_t rmsnorm_rope(T* x, long rows, long ld, int d, int parts, const float* gain0,
                        const float* gain1, const float2* rope, int L, int head_dim,
                        hipStream_t st);
// Patchify latents of the listed streams into rows [slot*L + tok][C*4].
template <typename T>
hipError_t patchify(const float* x, const int* slot_id, int n_slots, int cand_div, long D, int C,
                    int F, int H, int Wd, T* out, hipStream_t st);
// y[n] = sum_k W[n][k] * act(x[k]) + b[n]  (act: 0 none, 1 SiLU); fp32 out.
template <typename T>
hipError_t gemv(const T* W, const float* x, const float* b, int N, int K, int act, float* y,
                hipStream_t st);
// Sinusoidal timestep features [cos(1000 t w_k), sin(1000 t w_k)].
hipError_t time_features(float t, int freq_dim, float* out, hipStream_t st);
// mods[j][6][d] = m[6d] + table_j (tables at tables0 + j*table_stride);
// hmod[2][d] = e[d] + head_table.
hipError_t build_mods_strided(const float* m, const float* e, const float* tables0,
                              long table_stride, int n_blocks, const float* head_table, int d,
                              float* mods, float* hmod, hipStream_t st);
template <typename T> hipError_t cast_from_f32(const float* src, T* dst, long n, hipStream_t st);
// z[rows][d] += gate * y (gate: [d] or NULL for 1); d % 8 == 0.  Applies a
// stored attention-branch output y [rows][d] of the compute type.
template <typename T>
hipError_t residual_add(float* z, const T* y, const float* gate, long rows, int d, hipStream_t st);

// ---- cache rule, update, score (k_cache.hip)
struct DecideOut {     // written by the decision kernel, read back by the host
  int32_t n_compute;
  int32_t pad;
};
// Partial sums per (candidate, branch, chunk): sum (x - xref)^2 and sum xref^2.
int decide_chunks(long D);
hipError_t decide_partials(const float* x, const float* xref, int n_cand, int n_branch, long D,
                           double* partials, hipStream_t st);
// Finalize: per stream s = i*B + b, forced / rule / override -> mask, a_seen,
// compact list of computed streams and their branches, count.
// Streams (candidates x branches) one decision launch handles: 1024
// candidates with two branches each.
constexpr int MAX_DECIDE_STREAMS = 2048;
struct DecideParams {
  int n_streams, n_branch, step, n_steps, k_warm, k_cool, mode, static_k, nchunk;
  int use_partials, use_override;
  double tau;
};
hipError_t decide_finalize(const DecideParams& p, const double* partials, const uint8_t* override_mask,
                           double* a, uint8_t* has_ref, uint8_t* mask, double* a_seen,
                           int32_t* slot_list, int32_t* branch_list, DecideOut* out,
                           hipStream_t st);
// x_i += dt * cfg(v_i0, v_i1); v_ib = vbuf (computed) or x + delta (skipped);
// computed streams refresh delta and xref when store_state; the guided
// velocity is also written to vt_out when it is not NULL.
hipError_t cache_update(float* x, float* xref, float* delta, const float* vbuf,
                        const uint8_t* mask, int n_cand, int n_branch, long D, float dt,
                        float guidance, int store_state, float* vt_out, hipStream_t st);
int score_chunks(long D);
// Partial sums of <w, x_i - c * vt_i> per 8192-element chunk (vt NULL: <w, x_i>).
hipError_t score_partials(const float* x, const float* vt, float c, const float* w, int n_cand,
                          long D, double* partials, hipStream_t st);
hipError_t score_finalize(const double* partials, int n_cand, int nchunk, long D, double* scores,
                          hipStream_t st);

}  // namespace cs
