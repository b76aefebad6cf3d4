// Cache rule, fused skip/refresh/CFG/Euler update, and score reduction.
//
// Decision (Eq. indicator): per stream s = (candidate i, branch b) the drift
// ||x_i - xref_s||_F / ||xref_s||_F is accumulated into a_s; the call is
// skipped iff a_s <= tau, else it computes and a_s resets to 0.  The two
// sums are reduced in fp64, first per (candidate, 8192-element chunk) by a
// coalesced streaming kernel that reads x once for all branches, then per
// stream by one wave each (strided over the chunks, then a fixed butterfly),
// and a single wave takes the decisions and compacts the list of computing
// streams with a ballot (no atomics: results do not depend on timing).
//
// Update: skipped streams use x + Delta (Eq. skip); computed streams take
// the transformer output v and, when the cache is on, refresh Delta = v - x
// and xref = x (Eq. delta); branches are combined by Eq. cfg and the Euler
// step of Eq. euler is applied, all in one pass over the latents.
#include "kernels.hpp"

namespace cs {

constexpr int CHUNK_F4 = 8;                     // float4 per thread per chunk
constexpr int CHUNK = 256 * 4 * CHUNK_F4;       // 8192 elements

int decide_chunks(long D) { return cdiv(D, CHUNK); }
int score_chunks(long D) { return cdiv(D, CHUNK); }

// Block-wide fp64 sum in a fixed order (wave sums, then waves in order).
__device__ double block_sum(double v, double* sh) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh[wave] = v;
  __syncthreads();
  double t = 0.0;
  if (threadIdx.x == 0) t = ((sh[0] + sh[1]) + sh[2]) + sh[3];
  return t;
}

__global__ __launch_bounds__(256) void k_decide_partials(const float* __restrict__ x,
                                                          const float* __restrict__ xref,
                                                          int n_branch, long D,
                                                          double* __restrict__ partials) {
  __shared__ double sh[4];
  const int chunk = blockIdx.x, nchunk = gridDim.x, i = blockIdx.y;
  const long D4 = D >> 2;
  const float4* xi = reinterpret_cast<const float4*>(x + (long)i * D);
  double num[2] = {0.0, 0.0}, den[2] = {0.0, 0.0};
  for (int k = 0; k < CHUNK_F4; ++k) {
    const long j = (long)chunk * (CHUNK / 4) + k * 256 + threadIdx.x;
    if (j < D4) {
      const float4 xv = xi[j];
      for (int b = 0; b < n_branch; ++b) {
        const float4 r = reinterpret_cast<const float4*>(xref + ((long)i * n_branch + b) * D)[j];
        const float d0 = xv.x - r.x, d1 = xv.y - r.y, d2 = xv.z - r.z, d3 = xv.w - r.w;
        num[b] += ((double)d0 * d0 + (double)d1 * d1) + ((double)d2 * d2 + (double)d3 * d3);
        den[b] += ((double)r.x * r.x + (double)r.y * r.y) + ((double)r.z * r.z + (double)r.w * r.w);
      }
    }
  }
  for (int b = 0; b < n_branch; ++b) {
    const double tn = block_sum(num[b], sh);
    const double td = block_sum(den[b], sh);
    if (threadIdx.x == 0) {
      double* p = partials + (((long)i * n_branch + b) * nchunk + chunk) * 2;
      p[0] = tn;
      p[1] = td;
    }
  }
}

hipError_t decide_partials(const float* x, const float* xref, int n_cand, int n_branch, long D,
                           double* partials, hipStream_t st) {
  dim3 grid((unsigned)decide_chunks(D), (unsigned)n_cand);
  hipLaunchKernelGGL(k_decide_partials, grid, dim3(256), 0, st, x, xref, n_branch, D, partials);
  return hipGetLastError();
}

// Per-stream totals of the chunk partials, one wave per stream: lane l sums
// chunks l, l + 64, ... in order, then the lanes combine in a fixed butterfly
// (the order depends only on the chunk count, never on timing).
CS_DEV void wave_stream_sums(const double* __restrict__ ps, int nchunk, double& num, double& den) {
  const int lane = threadIdx.x & 63;
  double n = 0.0, d = 0.0;
  for (int c = lane; c < nchunk; c += 64) {
    const double2 v = reinterpret_cast<const double2*>(ps)[c];
    n += v.x;
    d += v.y;
  }
  num = wave_sum(n);
  den = wave_sum(d);
}

constexpr int FIN_WAVES = 16;

__global__ __launch_bounds__(64 * FIN_WAVES) void k_decide_finalize(DecideParams p,
                                                         const double* __restrict__ partials,
                                                         const uint8_t* __restrict__ ovr,
                                                         double* __restrict__ a,
                                                         uint8_t* __restrict__ has_ref,
                                                         uint8_t* __restrict__ mask,
                                                         double* __restrict__ a_seen,
                                                         int32_t* __restrict__ slots,
                                                         int32_t* __restrict__ branch,
                                                         DecideOut* __restrict__ out) {
  __shared__ double sums[2 * MAX_DECIDE_STREAMS];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (p.use_partials) {
    for (int s = wave; s < p.n_streams; s += FIN_WAVES) {
      double num, den;
      wave_stream_sums(partials + (long)s * p.nchunk * 2, p.nchunk, num, den);
      if (lane == 0) {
        sums[2 * s] = num;
        sums[2 * s + 1] = den;
      }
    }
  }
  __syncthreads();
  if (wave != 0) return;
  int count = 0;
  for (int base = 0; base < p.n_streams; base += 64) {
    const int s = base + lane;
    const bool valid = s < p.n_streams;
    bool compute = true;
    if (valid) {
      const bool forced = p.mode == 0 || p.step <= p.k_warm || p.step > p.n_steps - p.k_cool ||
                          !has_ref[s];
      double seen = __builtin_nan("");
      if (!forced) {
        if (p.mode == 2) {
          compute = ((p.step - p.k_warm) % p.static_k) == 0;
        } else if (p.use_partials) {
          const double num = sums[2 * s], den = sums[2 * s + 1];
          if (den > 0.0) {
            a[s] += sqrt(num) / sqrt(den);
            seen = a[s];
            compute = !(a[s] <= p.tau);
          }
        }
      }
      if (p.use_override) compute = ovr[s] != 0;
      if (compute) {
        a[s] = 0.0;
        has_ref[s] = 1;
      }
      mask[s] = compute ? 1 : 0;
      a_seen[s] = seen;
    }
    const unsigned long long bal = __ballot(valid && compute);
    const unsigned long long below = lane == 0 ? 0ull : (bal & ((1ull << lane) - 1ull));
    if (valid && compute) {
      slots[count + __popcll(below)] = s;
      branch[count + __popcll(below)] = s % p.n_branch;
    }
    count += __popcll(bal);
  }
  if (lane == 0) out->n_compute = count;
}

hipError_t decide_finalize(const DecideParams& p, const double* partials, const uint8_t* ovr,
                           double* a, uint8_t* has_ref, uint8_t* mask, double* a_seen,
                           int32_t* slots, int32_t* branch, DecideOut* out, hipStream_t st) {
  if (p.n_streams > MAX_DECIDE_STREAMS) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_decide_finalize, dim3(1), dim3(64 * FIN_WAVES), 0, st, p, partials, ovr, a, has_ref,
                     mask, a_seen, slots, branch, out);
  return hipGetLastError();
}

// One workgroup per (candidate, 1024 float4 of its latent): each thread
// handles UPD_F4 float4 spaced a workgroup apart (coalesced) and issues all
// of its loads before its stores.  The candidate and its branch masks are
// uniform per workgroup.  FULL: every element of the thread is in range
// (no per-element checks, so the loads are issued back to back).
constexpr int UPD_F4 = 4;

template <bool FULL>
__device__ __forceinline__ void cache_update_body(float4* __restrict__ xp, float* __restrict__ xref,
                                                  float* __restrict__ delta,
                                                  const float* __restrict__ vbuf, const int (&m)[2],
                                                  long s0, int n_branch, long D, long D4, long j0,
                                                  float dt, float w, int store_state,
                                                  float4* __restrict__ vtp) {
  auto in = [&](int k) { return FULL || j0 + k * 256 < D4; };
  float4 xv[UPD_F4], v[2][UPD_F4];
#pragma unroll
  for (int k = 0; k < UPD_F4; ++k)
    if (in(k)) xv[k] = xp[j0 + k * 256];
  // b runs to a compile-time bound so that v stays in registers
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    if (b >= n_branch) break;
    const long s = s0 + b;
    float4* dp = reinterpret_cast<float4*>(delta + s * D);
    if (m[b]) {
      const float4* vp = reinterpret_cast<const float4*>(vbuf + s * D);
#pragma unroll
      for (int k = 0; k < UPD_F4; ++k)
        if (in(k)) v[b][k] = vp[j0 + k * 256];
      if (store_state) {
        float4* rp = reinterpret_cast<float4*>(xref + s * D);
#pragma unroll
        for (int k = 0; k < UPD_F4; ++k) {
          if (!in(k)) continue;
          float4 dv;
          dv.x = v[b][k].x - xv[k].x; dv.y = v[b][k].y - xv[k].y;
          dv.z = v[b][k].z - xv[k].z; dv.w = v[b][k].w - xv[k].w;
          dp[j0 + k * 256] = dv;
          rp[j0 + k * 256] = xv[k];
        }
      }
    } else {
      float4 dv[UPD_F4];
#pragma unroll
      for (int k = 0; k < UPD_F4; ++k)
        if (in(k)) dv[k] = dp[j0 + k * 256];
#pragma unroll
      for (int k = 0; k < UPD_F4; ++k) {
        if (!in(k)) continue;
        v[b][k].x = xv[k].x + dv[k].x; v[b][k].y = xv[k].y + dv[k].y;
        v[b][k].z = xv[k].z + dv[k].z; v[b][k].w = xv[k].w + dv[k].w;
      }
    }
  }
#pragma unroll
  for (int k = 0; k < UPD_F4; ++k) {
    if (!in(k)) continue;
    float4 vt = v[0][k];
    if (n_branch == 2) {
      vt.x = v[1][k].x + w * (v[0][k].x - v[1][k].x);
      vt.y = v[1][k].y + w * (v[0][k].y - v[1][k].y);
      vt.z = v[1][k].z + w * (v[0][k].z - v[1][k].z);
      vt.w = v[1][k].w + w * (v[0][k].w - v[1][k].w);
    }
    float4 xn;
    xn.x = xv[k].x + dt * vt.x; xn.y = xv[k].y + dt * vt.y;
    xn.z = xv[k].z + dt * vt.z; xn.w = xv[k].w + dt * vt.w;
    xp[j0 + k * 256] = xn;
    if (vtp) vtp[j0 + k * 256] = vt;
  }
}

__global__ __launch_bounds__(256) void k_cache_update(float* __restrict__ x, float* __restrict__ xref,
                                                       float* __restrict__ delta,
                                                       const float* __restrict__ vbuf,
                                                       const uint8_t* __restrict__ mask, int n_cand,
                                                       int n_branch, long D, float dt, float w,
                                                       int store_state, float* __restrict__ vt_out) {
  const long D4 = D >> 2;
  const int i = blockIdx.y;
  const long s0 = (long)i * n_branch;
  const int m[2] = {mask[s0], n_branch == 2 ? (int)mask[s0 + 1] : 0};
  const long j0 = (long)blockIdx.x * (256 * UPD_F4) + threadIdx.x;
  float4* xp = reinterpret_cast<float4*>(x + (long)i * D);
  float4* vtp = vt_out ? reinterpret_cast<float4*>(vt_out + (long)i * D) : nullptr;
  if (j0 + (UPD_F4 - 1) * 256 < D4)
    cache_update_body<true>(xp, xref, delta, vbuf, m, s0, n_branch, D, D4, j0, dt, w, store_state, vtp);
  else
    cache_update_body<false>(xp, xref, delta, vbuf, m, s0, n_branch, D, D4, j0, dt, w, store_state, vtp);
}

hipError_t cache_update(float* x, float* xref, float* delta, const float* vbuf, const uint8_t* mask,
                        int n_cand, int n_branch, long D, float dt, float guidance,
                        int store_state, float* vt_out, hipStream_t st) {
  if (n_cand <= 0 || D <= 0) return hipSuccess;
  if (n_branch < 1 || n_branch > 2 || n_cand > 65535) return hipErrorInvalidValue;
  const dim3 grid((unsigned)cdiv(D >> 2, 256 * UPD_F4), (unsigned)n_cand);
  hipLaunchKernelGGL(k_cache_update, grid, dim3(256), 0, st, x, xref, delta, vbuf, mask, n_cand, n_branch,
                     D, dt, guidance, store_state, vt_out);
  return hipGetLastError();
}

// Partial sums of <w, x - c*vt> (vt NULL: <w, x>).
__global__ __launch_bounds__(256) void k_score_partials(const float* __restrict__ x,
                                                         const float* __restrict__ vt, float c,
                                                         const float* __restrict__ w, long D,
                                                         double* __restrict__ partials) {
  __shared__ double sh[4];
  const int chunk = blockIdx.x, nchunk = gridDim.x, i = blockIdx.y;
  const long D4 = D >> 2;
  const float4* xi = reinterpret_cast<const float4*>(x + (long)i * D);
  const float4* wv = reinterpret_cast<const float4*>(w);
  double acc = 0.0;
  for (int k = 0; k < CHUNK_F4; ++k) {
    const long j = (long)chunk * (CHUNK / 4) + k * 256 + threadIdx.x;
    if (j < D4) {
      float4 a = xi[j];
      const float4 b = wv[j];
      if (vt) {
        const float4 u = reinterpret_cast<const float4*>(vt + (long)i * D)[j];
        a.x -= c * u.x; a.y -= c * u.y; a.z -= c * u.z; a.w -= c * u.w;
      }
      acc += ((double)a.x * b.x + (double)a.y * b.y) + ((double)a.z * b.z + (double)a.w * b.w);
    }
  }
  const double t = block_sum(acc, sh);
  if (threadIdx.x == 0) partials[(long)i * nchunk + chunk] = t;
}

hipError_t score_partials(const float* x, const float* vt, float c, const float* w, int n_cand,
                          long D, double* partials, hipStream_t st) {
  dim3 grid((unsigned)score_chunks(D), (unsigned)n_cand);
  hipLaunchKernelGGL(k_score_partials, grid, dim3(256), 0, st, x, vt, c, w, D, partials);
  return hipGetLastError();
}

// One wave per candidate, the same fixed order as the decision totals.
__global__ __launch_bounds__(64) void k_score_finalize(const double* __restrict__ partials,
                                                       int nchunk, double inv_sqrt_d,
                                                       double* __restrict__ scores) {
  const int i = blockIdx.x, lane = threadIdx.x;
  const double* ps = partials + (long)i * nchunk;
  double s = 0.0;
  for (int c = lane; c < nchunk; c += 64) s += ps[c];
  s = wave_sum(s);
  if (lane == 0) scores[i] = s * inv_sqrt_d;
}

hipError_t score_finalize(const double* partials, int n_cand, int nchunk, long D, double* scores,
                          hipStream_t st) {
  if (n_cand <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_score_finalize, dim3((unsigned)n_cand), dim3(64), 0, st, partials, nchunk,
                     1.0 / sqrt((double)D), scores);
  return hipGetLastError();
}

}  // namespace cs
