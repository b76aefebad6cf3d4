// Row-wise and small kernels: layer norm with adaLN modulation, RMSNorm with
// 3D RoPE, patchify, GEMV for the timestep MLP, modulation tables, casts.
// All are bandwidth- or latency-bound; one wave per row, reductions in fp32
// over the row in a fixed lane/step order.
#include "kernels.hpp"

namespace cs {

// ---------------------------------------------------------------- layer norm
// One wave per row.  Three passes over the row (mean, centred variance,
// write), the repeats served from cache.
template <typename T>
__global__ __launch_bounds__(256) void k_layer_norm(const float* __restrict__ z, long rows, int d,
                                                     const float* __restrict__ p0,
                                                     const float* __restrict__ p1, int mode,
                                                     T* __restrict__ u) {
  const long row = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const float4* zr = reinterpret_cast<const float4*>(z + row * d);
  const int n4 = d >> 2;
  float s = 0.0f;
  for (int c = lane; c < n4; c += 64) {
    float4 v = zr[c];
    s += (v.x + v.y) + (v.z + v.w);
  }
  const float mean = wave_sum(s) / (float)d;
  float q = 0.0f;
  for (int c = lane; c < n4; c += 64) {
    float4 v = zr[c];
    float a = v.x - mean, b = v.y - mean, e = v.z - mean, f = v.w - mean;
    q += (a * a + b * b) + (e * e + f * f);
  }
  const float rstd = 1.0f / sqrtf(wave_sum(q) / (float)d + 1e-6f);
  T* ur = u + row * d;
  for (int c = lane; c < n4; c += 64) {
    float4 v = zr[c];
    float in[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int col = 4 * c + k;
      const float nv = (in[k] - mean) * rstd;
      const float y = mode == 0 ? nv * (1.0f + p1[col]) + p0[col] : nv * p0[col] + p1[col];
      ur[col] = to_t<T>(y);
    }
  }
}

template <typename T>
hipError_t layer_norm_mod(const float* z, long rows, int d, const float* p0, const float* p1,
                          int mode, T* u, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_layer_norm<T>, dim3((unsigned)cdiv(rows, 4)), dim3(256), 0, st, z, rows, d,
                     p0, p1, mode, u);
  return hipGetLastError();
}

// ------------------------------------------------------------ RMSNorm + RoPE
// One wave per (row, part).  RoPE pairs are adjacent channels (2p, 2p+1) of
// a head; the table holds (cos, sin) per token and pair.
template <typename T>
__global__ __launch_bounds__(256) void k_rmsnorm_rope(T* __restrict__ x, long rows, long ld, int d,
                                                       int parts, const float* __restrict__ g0,
                                                       const float* __restrict__ g1,
                                                       const float2* __restrict__ rope, int L,
                                                       int head_dim) {
  const long item = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (item >= rows * parts) return;
  const long row = item / parts;
  const int part = (int)(item - row * parts);
  T* xr = x + row * ld + (long)part * d;
  const float* g = part == 0 ? g0 : g1;
  const int npair = d >> 1;
  float s = 0.0f;
  for (int p = lane; p < npair; p += 64) {
    const float a = to_f(xr[2 * p]), b = to_f(xr[2 * p + 1]);
    s += a * a + b * b;
  }
  const float r = 1.0f / sqrtf(wave_sum(s) / (float)d + 1e-6f);
  const int tok = (int)(row % L);
  const int hp = head_dim >> 1;
  for (int p = lane; p < npair; p += 64) {
    float a = to_f(xr[2 * p]) * r * g[2 * p];
    float b = to_f(xr[2 * p + 1]) * r * g[2 * p + 1];
    if (rope) {
      const float2 cs_ = rope[(long)tok * hp + (p % hp)];
      const float na = a * cs_.x - b * cs_.y;
      const float nb = a * cs_.y + b * cs_.x;
      a = na;
      b = nb;
    }
    xr[2 * p] = to_t<T>(a);
    xr[2 * p + 1] = to_t<T>(b);
  }
}

template <typename T>
hipError_t rmsnorm_rope(T* x, long rows, long ld, int d, int parts, const float* g0,
                        const float* g1, const float2* rope, int L, int head_dim, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_rmsnorm_rope<T>, dim3((unsigned)cdiv(rows * parts, 4)), dim3(256), 0, st, x,
                     rows, ld, d, parts, g0, g1, rope, L, head_dim);
  return hipGetLastError();
}

// ------------------------------------------------------------------ patchify
// Thread per (slot, token, channel): the 2x2 patch of channel c at token
// (f, h, w) becomes columns c*4 + dy*2 + dx of row slot*L + token.
template <typename T>
__global__ __launch_bounds__(256) void k_patchify(const float* __restrict__ x,
                                                   const int* __restrict__ slot_id, int n_slots,
                                                   int cand_div, long D, int C, int F, int H,
                                                   int Wd, T* __restrict__ out) {
  const int gh = H / 2, gw = Wd / 2;
  const long L = (long)F * gh * gw;
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)n_slots * L * C) return;
  const int c = (int)(idx % C);
  const long rt = idx / C;
  const int s = (int)(rt / L);
  const long tok = rt - (long)s * L;
  const int f = (int)(tok / (gh * gw));
  const int rem = (int)(tok - (long)f * gh * gw);
  const int hh = rem / gw, ww = rem - hh * gw;
  const int cand = slot_id[s] / cand_div;
  const float* src = x + (long)cand * D + (((long)c * F + f) * H + 2 * hh) * Wd + 2 * ww;
  T* dst = out + rt * (long)(C * 4) + c * 4;
  dst[0] = to_t<T>(src[0]);
  dst[1] = to_t<T>(src[1]);
  dst[2] = to_t<T>(src[Wd]);
  dst[3] = to_t<T>(src[Wd + 1]);
}

template <typename T>
hipError_t patchify(const float* x, const int* slot_id, int n_slots, int cand_div, long D, int C,
                    int F, int H, int Wd, T* out, hipStream_t st) {
  const long n = (long)n_slots * F * (H / 2) * (Wd / 2) * C;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_patchify<T>, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, st, x, slot_id,
                     n_slots, cand_div, D, C, F, H, Wd, out);
  return hipGetLastError();
}

// ---------------------------------------------------------------------- GEMV
// One wave per output; the input vector (after the optional SiLU) is staged
// in LDS once per workgroup.
template <typename T>
__global__ __launch_bounds__(256) void k_gemv(const T* __restrict__ W, const float* __restrict__ x,
                                               const float* __restrict__ b, int N, int K, int act,
                                               float* __restrict__ y) {
  extern __shared__ float sx[];
  for (int k = threadIdx.x; k < K; k += 256) {
    const float v = x[k];
    sx[k] = act == 1 ? silu(v) : v;
  }
  __syncthreads();
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (n >= N) return;
  const T* wr = W + (long)n * K;
  float s = 0.0f;
  for (int k = lane; k < K; k += 64) s += to_f(wr[k]) * sx[k];
  s = wave_sum(s);
  if (lane == 0) y[n] = s + (b ? b[n] : 0.0f);
}

template <typename T>
hipError_t gemv(const T* W, const float* x, const float* b, int N, int K, int act, float* y,
                hipStream_t st) {
  hipLaunchKernelGGL(k_gemv<T>, dim3((unsigned)cdiv(N, 4)), dim3(256), (size_t)K * sizeof(float),
                     st, W, x, b, N, K, act, y);
  return hipGetLastError();
}

// ---------------------------------------------------------- time features
__global__ void k_time_features(float t, int half, float* out) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= half) return;
  // frequency 10000^(-k/half); the angle is formed in double so that the
  // fp32 features are correctly rounded for large 1000*t*w.
  const double om = exp(-log(10000.0) * (double)k / (double)half);
  const double arg = 1000.0 * (double)t * om;
  out[k] = (float)cos(arg);
  out[half + k] = (float)sin(arg);
}

hipError_t time_features(float t, int freq_dim, float* out, hipStream_t st) {
  const int half = freq_dim / 2;
  hipLaunchKernelGGL(k_time_features, dim3((unsigned)cdiv(half, 128)), dim3(128), 0, st, t, half,
                     out);
  return hipGetLastError();
}

// --------------------------------------------------------- modulation tables
__global__ void k_build_mods(const float* __restrict__ m, const float* __restrict__ e,
                             const float* __restrict__ tables0, long stride, int n_blocks,
                             const float* __restrict__ head_table, int d, float* __restrict__ mods,
                             float* __restrict__ hmod) {
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  const long per = 6L * d;
  if (idx < per * n_blocks) {
    const int j = (int)(idx / per);
    const long r = idx - (long)j * per;
    mods[idx] = m[r] + tables0[(long)j * stride + r];
  } else if (idx < per * n_blocks + 2L * d) {
    const long r = idx - per * n_blocks;
    hmod[r] = e[r % d] + head_table[r];
  }
}

hipError_t build_mods_strided(const float* m, const float* e, const float* tables0,
                              long table_stride, int n_blocks, const float* head_table, int d,
                              float* mods, float* hmod, hipStream_t st) {
  const long n = 6L * d * n_blocks + 2L * d;
  hipLaunchKernelGGL(k_build_mods, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, st, m, e, tables0,
                     table_stride, n_blocks, head_table, d, mods, hmod);
  return hipGetLastError();
}

// ------------------------------------------------------------------- casts
template <typename T>
__global__ void k_cast(const float* __restrict__ s, T* __restrict__ d, long n) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i < n) d[i] = to_t<T>(s[i]);
}

template <typename T> hipError_t cast_from_f32(const float* src, T* dst, long n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_cast<T>, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, st, src, dst, n);
  return hipGetLastError();
}

#define CS_INST(T)                                                                              \
  template hipError_t layer_norm_mod<T>(const float*, long, int, const float*, const float*,   \
                                        int, T*, hipStream_t);                                  \
  template hipError_t rmsnorm_rope<T>(T*, long, long, int, int, const float*, const float*,    \
                                      const float2*, int, int, hipStream_t);                    \
  template hipError_t patchify<T>(const float*, const int*, int, int, long, int, int, int, int, \
                                  T*, hipStream_t);                                             \
  template hipError_t gemv<T>(const T*, const float*, const float*, int, int, int, float*,     \
                              hipStream_t);                                                     \
  template hipError_t cast_from_f32<T>(const float*, T*, long, hipStream_t);
CS_INST(bf16)
CS_INST(float)
#undef CS_INST

}  // namespace cs
