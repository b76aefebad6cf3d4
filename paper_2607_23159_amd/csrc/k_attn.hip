// Attention launchers: tile shapes per element type and head size.
#include "attn_kernel.hpp"

namespace cs {

int attn_kv_tile(int dtype_bytes, int head_dim) {
  if (dtype_bytes == 2) return 64;
  return head_dim > 64 ? 32 : 64;
}

template <typename T, int DH, int QB, int KVT, int NW, int OCC>
static hipError_t launch_flash(const AttnArgs<T>& a, hipStream_t st) {
  const int qpw = NW * QB * 32;
  const long nwg = (long)cdiv(a.lq, qpw) * a.heads * a.n_streams;
  if (nwg * 64 * NW > 0xFFFFFFFFL) return hipErrorInvalidConfiguration;
  dim3 grid((unsigned)nwg);
  if (a.kv_sel)
    hipLaunchKernelGGL((k_flash<T, DH, QB, KVT, NW, OCC, true>), grid, dim3(64 * NW), 0, st, a);
  else
    hipLaunchKernelGGL((k_flash<T, DH, QB, KVT, NW, OCC, false>), grid, dim3(64 * NW), 0, st, a);
  return hipGetLastError();
}

// bf16, head dim 32: XOR-swizzled direct-to-LDS tiles of 64 keys in a
// 4-deep ring, one 32-query block per wave.
template <int DH, int QB, int NW, int OCC>
static hipError_t launch_flash_dl(const AttnArgs<bf16>& a, hipStream_t st) {
  constexpr int KVT = 64, STAGES = 4;
  const long nwg = (long)cdiv(a.lq, NW * QB * 32) * a.heads * a.n_streams;
  if (nwg * 64 * NW > 0xFFFFFFFFL) return hipErrorInvalidConfiguration;
  // buffer ranges and offsets are 32-bit byte counts
  if ((long)a.lk * a.k_ld * 2 > 0x7FFFFFFFL || (long)DH * a.vt_ld * 2 > 0x7FFFFFFFL)
    return hipErrorInvalidValue;
  if (a.vt_ld < round_up(a.lk, KVT)) return hipErrorInvalidValue;
  if (a.kv_sel)
    hipLaunchKernelGGL((k_flash_dl<DH, QB, KVT, NW, OCC, STAGES, true>), dim3((unsigned)nwg),
                       dim3(64 * NW), 0, st, a);
  else
    hipLaunchKernelGGL((k_flash_dl<DH, QB, KVT, NW, OCC, STAGES, false>), dim3((unsigned)nwg),
                       dim3(64 * NW), 0, st, a);
  return hipGetLastError();
}

// bf16, head dims 64 and 128: padded-row tiles of 64 keys in a 3-deep ring
// (105 KB of LDS at 128: one workgroup per CU), 32 queries per wave.  Twelve
// waves (three per SIMD) are the faster shape per query; eight waves (two per
// SIMD) take 256 instead of 384 queries per workgroup, which matters when the
// grid is a few rounds of the CUs long: at one 32,760-token stream of 12 heads,
// 1032 twelve-wave workgroups fill 256 CUs 4.03 times (five rounds) while 1536
// eight-wave ones fill them exactly six times.  Each wave's arithmetic is the
// same in both shapes (same key order, same per-wave rescale decisions), so
// the outputs are bitwise equal and the choice never changes a result.
static int cu_count() {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cus[dev] <= 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cus[dev] = n;
  }
  return cus[dev];
}

template <int DH, int NW, int OCC>
static hipError_t launch_flash_pad_nw(const AttnArgs<bf16>& a, hipStream_t st) {
  constexpr int STAGES = 3;
  const long nwg = (long)cdiv(a.lq, NW * 32) * a.heads * a.n_streams;
  if (nwg * 64 * NW > 0xFFFFFFFFL) return hipErrorInvalidConfiguration;
  if (a.kv_sel)
    hipLaunchKernelGGL((k_flash_pad<DH, NW, OCC, STAGES, true>), dim3((unsigned)nwg), dim3(64 * NW), 0,
                       st, a);
  else
    hipLaunchKernelGGL((k_flash_pad<DH, NW, OCC, STAGES, false>), dim3((unsigned)nwg), dim3(64 * NW), 0,
                       st, a);
  return hipGetLastError();
}

template <int DH>
static hipError_t launch_flash_pad(const AttnArgs<bf16>& a, hipStream_t st) {
  if ((long)a.lk * a.k_ld * 2 > 0x7FFFFFFFL || (long)DH * a.vt_ld * 2 > 0x7FFFFFFFL)
    return hipErrorInvalidValue;
  // every 64-key tile of V^T must lie inside its padded row
  if (a.vt_ld < round_up(a.lk, 64)) return hipErrorInvalidValue;
  // estimated time in rounds of the CUs x queries per workgroup; eight waves
  // run about 3.5% slower per query than twelve
  const long cus = cu_count(), sh = (long)a.heads * a.n_streams;
  const double t12 = (double)cdiv(cdiv(a.lq, 384) * sh, cus) * 384.0;
  const double t8 = (double)cdiv(cdiv(a.lq, 256) * sh, cus) * 256.0 * 1.035;
  if (t8 < t12) return launch_flash_pad_nw<DH, 8, 2>(a, st);
  return launch_flash_pad_nw<DH, 12, 3>(a, st);
}

template <>
hipError_t flash_attention<bf16>(const AttnArgs<bf16>& a, int head_dim, hipStream_t st) {
  if (a.lq <= 0 || a.n_streams <= 0) return hipSuccess;
  switch (head_dim) {
    case 128: return launch_flash_pad<128>(a, st);
    case 64: return launch_flash_pad<64>(a, st);
    case 32: return launch_flash_dl<32, 1, 4, 1>(a, st);
    default: return hipErrorInvalidValue;
  }
}

template <>
hipError_t flash_attention<float>(const AttnArgs<float>& a, int head_dim, hipStream_t st) {
  if (a.lq <= 0 || a.n_streams <= 0) return hipSuccess;
  switch (head_dim) {
    case 128: return launch_flash<float, 128, 1, 32, 4, 1>(a, st);
    case 64: return launch_flash<float, 64, 1, 64, 4, 1>(a, st);
    case 32: return launch_flash<float, 32, 1, 64, 4, 1>(a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace cs
