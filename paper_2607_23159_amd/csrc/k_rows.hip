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

// Register-resident variant: the row (d = NV * 256) is read once as float4
// chunks (lane-contiguous, so each wave access is 1 KB), reduced twice from
// registers and written with one 8- or 16-byte store per chunk.
template <typename T, int NV>
__global__ __launch_bounds__(256) void k_layer_norm_reg(const float* __restrict__ z, long rows,
                                                         int d, const float* __restrict__ p0,
                                                         const float* __restrict__ p1, int mode,
                                                         T* __restrict__ u) {
  const long row = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const float4* zr = reinterpret_cast<const float4*>(z + row * d);
  float4 v[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k) v[k] = zr[k * 64 + lane];
  float s = 0.0f;
#pragma unroll
  for (int k = 0; k < NV; ++k) s += (v[k].x + v[k].y) + (v[k].z + v[k].w);
  const float mean = wave_sum(s) / (float)d;
  float q = 0.0f;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const float a = v[k].x - mean, b = v[k].y - mean, e = v[k].z - mean, f = v[k].w - mean;
    q += (a * a + b * b) + (e * e + f * f);
  }
  const float rstd = 1.0f / sqrtf(wave_sum(q) / (float)d + 1e-6f);
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int col = 4 * (k * 64 + lane);
    const float4 a = *reinterpret_cast<const float4*>(p0 + col);
    const float4 b = *reinterpret_cast<const float4*>(p1 + col);
    const float in[4] = {v[k].x, v[k].y, v[k].z, v[k].w};
    const float pa[4] = {a.x, a.y, a.z, a.w}, pb[4] = {b.x, b.y, b.z, b.w};
    float y[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float nv = (in[r] - mean) * rstd;
      y[r] = mode == 0 ? nv * (1.0f + pb[r]) + pa[r] : nv * pa[r] + pb[r];
    }
    T* dst = u + row * d + col;
    if constexpr (sizeof(T) == 2) {
      bf16x4 o;
#pragma unroll
      for (int r = 0; r < 4; ++r) o[r] = to_t<T>(y[r]);
      *reinterpret_cast<bf16x4*>(dst) = o;
    } else {
      *reinterpret_cast<float4*>(dst) = make_float4(y[0], y[1], y[2], y[3]);
    }
  }
}

template <typename T>
hipError_t layer_norm_mod(const float* z, long rows, int d, const float* p0, const float* p1,
                          int mode, T* u, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  const dim3 grid((unsigned)cdiv(rows, 4)), block(256);
  switch (d % 256 == 0 ? d / 256 : 0) {
#define CS_LN(NV) \
  case NV: hipLaunchKernelGGL((k_layer_norm_reg<T, NV>), grid, block, 0, st, z, rows, d, p0, p1, mode, u); break;
    CS_LN(1) CS_LN(2) CS_LN(3) CS_LN(4) CS_LN(6) CS_LN(8) CS_LN(12) CS_LN(16) CS_LN(20) CS_LN(24)
#undef CS_LN
    default:
      hipLaunchKernelGGL(k_layer_norm<T>, grid, block, 0, st, z, rows, d, p0, p1, mode, u);
  }
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

// Register-resident variant: lane owns NV chunks of 8 consecutive channels
// (4 RoPE pairs, 16 bytes in bf16); one read, one write per chunk.
template <typename T> struct Vec8;
template <> struct Vec8<bf16> {
  typedef bf16x8 V;
  static CS_DEV void get(const bf16* p, float* f) {
    const bf16x8 v = *reinterpret_cast<const bf16x8*>(p);
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = (float)v[i];
  }
  static CS_DEV void put(bf16* p, const float* f) {
    bf16x8 v;
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = (bf16)f[i];
    *reinterpret_cast<bf16x8*>(p) = v;
  }
};
template <> struct Vec8<float> {
  static CS_DEV void get(const float* p, float* f) {
    const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w; f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
  }
  static CS_DEV void put(float* p, const float* f) {
    reinterpret_cast<float4*>(p)[0] = make_float4(f[0], f[1], f[2], f[3]);
    reinterpret_cast<float4*>(p)[1] = make_float4(f[4], f[5], f[6], f[7]);
  }
};

template <typename T, int NV>
__global__ __launch_bounds__(256) void k_rmsnorm_rope_reg(T* __restrict__ x, long rows, long ld,
                                                           int d, int parts,
                                                           const float* __restrict__ g0,
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
  float v[NV][8];
#pragma unroll
  for (int k = 0; k < NV; ++k) Vec8<T>::get(xr + 8 * (k * 64 + lane), v[k]);
  float s = 0.0f;
#pragma unroll
  for (int k = 0; k < NV; ++k)
#pragma unroll
    for (int i = 0; i < 8; ++i) s += v[k][i] * v[k][i];
  const float r = 1.0f / sqrtf(wave_sum(s) / (float)d + 1e-6f);
  const int tok = (int)(row % L);
  const int hp = head_dim >> 1;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int c0 = 8 * (k * 64 + lane);
    const float4 ga = *reinterpret_cast<const float4*>(g + c0);
    const float4 gb = *reinterpret_cast<const float4*>(g + c0 + 4);
    const float gg[8] = {ga.x, ga.y, ga.z, ga.w, gb.x, gb.y, gb.z, gb.w};
    float y[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) y[i] = v[k][i] * r * gg[i];
    if (rope) {
      const float4* t = reinterpret_cast<const float4*>(rope + (long)tok * hp + ((c0 >> 1) % hp));
      const float4 t0 = t[0], t1 = t[1];
      const float cs_[8] = {t0.x, t0.y, t0.z, t0.w, t1.x, t1.y, t1.z, t1.w};
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const float a = y[2 * p], b = y[2 * p + 1], c = cs_[2 * p], sn = cs_[2 * p + 1];
        y[2 * p] = a * c - b * sn;
        y[2 * p + 1] = a * sn + b * c;
      }
    }
    Vec8<T>::put(xr + c0, y);
  }
}

template <typename T>
hipError_t rmsnorm_rope(T* x, long rows, long ld, int d, int parts, const float* g0,
                        const float* g1, const float2* rope, int L, int head_dim, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  const dim3 grid((unsigned)cdiv(rows * parts, 4)), block(256);
  switch (d % 512 == 0 ? d / 512 : 0) {
#define CS_RR(NV)                                                                                \
  case NV:                                                                                       \
    hipLaunchKernelGGL((k_rmsnorm_rope_reg<T, NV>), grid, block, 0, st, x, rows, ld, d, parts, g0, \
                       g1, rope, L, head_dim);                                                   \
    break;
    CS_RR(1) CS_RR(2) CS_RR(3) CS_RR(4) CS_RR(6) CS_RR(8) CS_RR(10) CS_RR(12)
#undef CS_RR
    default:
      hipLaunchKernelGGL(k_rmsnorm_rope<T>, grid, block, 0, st, x, rows, ld, d, parts, g0, g1, rope,
                         L, head_dim);
  }
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

// ------------------------------------------------ stored-output reuse
// z[r][c] += gate[c] * y[r][c] (gate NULL: 1), 8 consecutive channels per
// thread: the residual update of an attention branch whose stored output is
// reused instead of recomputed.
template <typename T>
__global__ __launch_bounds__(256) void k_residual_add(float* __restrict__ z, const T* __restrict__ y,
                                                      const float* __restrict__ gate, long n8,
                                                      int d8) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= n8) return;
  float yv[8], zv[8];
  Vec8<T>::get(y + i * 8, yv);
  Vec8<float>::get(z + i * 8, zv);
  if (gate) {
    float g[8];
    Vec8<float>::get(gate + (i % d8) * 8, g);
#pragma unroll
    for (int r = 0; r < 8; ++r) zv[r] += g[r] * yv[r];
  } else {
#pragma unroll
    for (int r = 0; r < 8; ++r) zv[r] += yv[r];
  }
  Vec8<float>::put(z + i * 8, zv);
}

template <typename T>
hipError_t residual_add(float* z, const T* y, const float* gate, long rows, int d, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  if (d % 8 != 0) return hipErrorInvalidValue;
  const long n8 = rows * d / 8;
  hipLaunchKernelGGL(k_residual_add<T>, dim3((unsigned)cdiv(n8, 256)), dim3(256), 0, st, z, y, gate,
                     n8, d / 8);
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
  template hipError_t cast_from_f32<T>(const float*, T*, long, hipStream_t);                 \
  template hipError_t residual_add<T>(float*, const T*, const float*, long, int, hipStream_t);
CS_INST(bf16)
CS_INST(float)
#undef CS_INST

}  // namespace cs
