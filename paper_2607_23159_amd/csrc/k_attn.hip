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
// (105 KB of LDS at 128), 12 waves of 32 queries (three per SIMD).
template <int DH>
static hipError_t launch_flash_pad(const AttnArgs<bf16>& a, hipStream_t st) {
  constexpr int NW = 12, OCC = 3, STAGES = 3;
  const long nwg = (long)cdiv(a.lq, NW * 32) * a.heads * a.n_streams;
  if (nwg * 64 * NW > 0xFFFFFFFFL) return hipErrorInvalidConfiguration;
  if ((long)a.lk * a.k_ld * 2 > 0x7FFFFFFFL || (long)DH * a.vt_ld * 2 > 0x7FFFFFFFL)
    return hipErrorInvalidValue;
  // every 64-key tile of V^T must lie inside its padded row
  if (a.vt_ld < round_up(a.lk, 64)) return hipErrorInvalidValue;
  if (a.kv_sel)
    hipLaunchKernelGGL((k_flash_pad<DH, NW, OCC, STAGES, true>), dim3((unsigned)nwg), dim3(64 * NW), 0,
                       st, a);
  else
    hipLaunchKernelGGL((k_flash_pad<DH, NW, OCC, STAGES, false>), dim3((unsigned)nwg), dim3(64 * NW), 0,
                       st, a);
  return hipGetLastError();
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
