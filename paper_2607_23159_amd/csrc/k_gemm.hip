// GEMM launchers: tile shapes per element type and the fused epilogues.
#include "gemm_kernel.hpp"

namespace cs {

// ------------------------------------------------------------- launchers
// bf16: direct-to-LDS kernels on 16x16x32 MFMAs, 256x256 tiles, K slices of
//       64, tile groups of 4 tile-rows: k_gemm_w4 (4 waves of 128x128, one
//       per SIMD) and, for residual updates at short K, k_gemm_dl (8 waves
//       of 128x64, two per SIMD).  Both sum in the same order (bitwise
//       equal results).  K must be a multiple of 64.
// fp32: register-staged kernel, 128x128 tiles, 4 waves of 64x64, K slices of 16.
// Narrow N (head GEMM, N = patch_dim): register-staged 128x64 tiles.
template <typename T> struct GemmCfg;
template <> struct GemmCfg<float> {
  static constexpr int BM = 128, BN = 128, BK = 16, WM = 64, WN = 64, NW = 4, OCC = 1, GM = 1;
};
template <typename T> struct GemmCfgNarrow;
template <> struct GemmCfgNarrow<bf16> {
  static constexpr int BM = 128, BN = 64, BK = 32, WM = 32, WN = 64, NW = 4, OCC = 1, GM = 1;
};
template <> struct GemmCfgNarrow<float> {
  static constexpr int BM = 128, BN = 64, BK = 16, WM = 32, WN = 64, NW = 4, OCC = 1, GM = 1;
};
struct DlCfg {
  static constexpr int BM = 256, BN = 256, BK = 64, WM = 128, WN = 64, NW = 8, OCC = 2, ST = 2,
                       GM = 4;
};

// ------------------------------------------------------- weight tiling
// bf16 weights for the direct-load kernel: [N][K] fp32 row-major ->
// blocks of DlCfg::BN rows x DlCfg::BK columns, block (tn, kt) at
// ((tn * K/BK + kt) * BN * BK) elements; inside a block row r holds its 8
// chunks of 8 columns with logical chunk c at physical position
// c ^ gemm_swz(r), the LDS layout of the kernel.  Rows past N are zero.
__global__ __launch_bounds__(256) void k_tile_weight(const float* __restrict__ src, int N, int K,
                                                     bf16* __restrict__ dst, long n_chunks) {
  constexpr int BN = DlCfg::BN, BK = DlCfg::BK, CPR = BK / 8;
  const long q = (long)blockIdx.x * 256 + threadIdx.x;
  if (q >= n_chunks) return;
  const long blk = q / (BN * CPR);
  const int within = (int)(q - blk * BN * CPR);
  const int r = within / CPR, p = within % CPR;
  const int nk = K / BK;
  const int tn = (int)(blk / nk), kt = (int)(blk % nk);
  const int n = tn * BN + r;
  const int k0 = kt * BK + (p ^ gemm_swz(r)) * 8;
  bf16x8 v;
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = n < N ? (bf16)src[(long)n * K + k0 + e] : (bf16)0.0f;
  *reinterpret_cast<bf16x8*>(dst + q * 8) = v;
}

long gemm_tiled_weight_elems(int N, int K) { return round_up(N, DlCfg::BN) * (long)K; }

hipError_t gemm_tile_weight(const float* src, int N, int K, bf16* dst, hipStream_t st) {
  if (N <= 0 || K % DlCfg::BK != 0) return hipErrorInvalidValue;
  const long n_chunks = gemm_tiled_weight_elems(N, K) / 8;
  hipLaunchKernelGGL(k_tile_weight, dim3((unsigned)cdiv(n_chunks, 256)), dim3(256), 0, st, src, N, K, dst,
                     n_chunks);
  return hipGetLastError();
}

template <typename T, class C, class Epi>
static hipError_t launch_staged(const T* A, long lda, const T* W, long ldw, int M, int N, int K,
                                Epi epi, hipStream_t st) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (K <= 0 || K % C::BK != 0 || N % 4 != 0) return hipErrorInvalidValue;
  const long tiles = (long)cdiv(M, C::BM) * cdiv(N, C::BN);
  hipLaunchKernelGGL((k_gemm<T, C::BM, C::BN, C::BK, C::WM, C::WN, C::NW, C::OCC, C::GM, Epi>),
                     dim3((unsigned)tiles), dim3(64 * C::NW), 0, st, A, lda, W, ldw, M, N, K, epi);
  return hipGetLastError();
}

// Residual-update epilogues read and write the fp32 residual stream: at
// short K their epilogue, not the products, sets the pace, and eight waves
// per CU (k_gemm_dl) keep more of those reads in flight than four.  Measured
// crossover: k_gemm_dl is 8% faster at K = 1536 and 2% at K = 3072, k_gemm_w4
// 4% faster at K = 5120 and 9% at K = 14336.
template <class Epi> struct EpiIsResidual : std::false_type {};
template <int G> struct EpiIsResidual<EpiResidual<G>> : std::true_type {};
template <int G, typename T> struct EpiIsResidual<EpiResidualStore<G, T>> : std::true_type {};
constexpr int W4_MIN_RESIDUAL_K = 4096;

template <typename T, class Epi>
static hipError_t launch(const T* A, long lda, const T* W, long ldw, int M, int N, int K, Epi epi,
                         hipStream_t st) {
  if constexpr (sizeof(T) == 2) {
    typedef DlCfg C;
    if (M <= 0 || N <= 0) return hipSuccess;
    if (K <= 0 || K % C::BK != 0 || N % 4 != 0) return hipErrorInvalidValue;
    // W is pre-tiled (row stride K); per-tile buffer ranges are 32-bit byte counts
    if (ldw != K) return hipErrorInvalidValue;
    if ((long)std::max(C::BM, C::BN) * std::max(lda, (long)K) * 2 > 0x7FFFFFFFL) return hipErrorInvalidValue;
    const long tiles = (long)cdiv(M, C::BM) * cdiv(N, C::BN);
    if (EpiIsResidual<Epi>::value && K < W4_MIN_RESIDUAL_K) {
      hipLaunchKernelGGL((k_gemm_dl<C::BM, C::BN, C::BK, C::WM, C::WN, C::NW, C::OCC, C::ST, C::GM, Epi>),
                         dim3((unsigned)tiles), dim3(64 * C::NW), 0, st, A, lda, W, ldw, M, N, K, epi);
    } else {
      constexpr int PD = EpiIsResidual<Epi>::value ? 8 : 2;
      hipLaunchKernelGGL((k_gemm_w4<C::BM, C::GM, PD, Epi>), dim3((unsigned)tiles), dim3(256), 0, st, A,
                         lda, W, ldw, M, N, K, epi);
    }
    return hipGetLastError();
  } else {
    return launch_staged<T, GemmCfg<T>>(A, lda, W, ldw, M, N, K, epi, st);
  }
}

template <typename T>
hipError_t gemm_store(const T* A, long lda, const T* W, int M, int N, int K, const float* bias,
                      int act, T* out, long ldo, hipStream_t st) {
  if (!bias) return hipErrorInvalidValue;
  if (act == 1) return launch<T>(A, lda, W, K, M, N, K, EpiStore<T, 1>{out, ldo, bias}, st);
  return launch<T>(A, lda, W, K, M, N, K, EpiStore<T, 0>{out, ldo, bias}, st);
}

template <typename T>
hipError_t gemm_store_t(const T* A, long lda, const T* W, int M, int N, int K, const float* bias,
                        T* out, long ldo, hipStream_t st) {
  EpiStoreT<T> e{out, ldo, bias};
  return launch<T>(A, lda, W, K, M, N, K, e, st);
}

template <typename T>
hipError_t gemm_qkv(const T* A, const T* W, int M, int d, const float* bias, int L, T* qk, T* vt,
                    long vt_ld, hipStream_t st) {
  EpiQKV<T> e{qk, vt, bias, d, L, vt_ld, (long)d * vt_ld};
  return launch<T>(A, d, W, d, M, 3 * d, d, e, st);
}

template <typename T>
hipError_t gemm_residual(const T* A, long lda, const T* W, int M, int N, int K, const float* bias,
                         const float* gate, float* z, T* y, hipStream_t st) {
  if (!bias) return hipErrorInvalidValue;
  if (y) {
    if (gate) return launch<T>(A, lda, W, K, M, N, K, EpiResidualStore<1, T>{z, N, bias, gate, y}, st);
    return launch<T>(A, lda, W, K, M, N, K, EpiResidualStore<0, T>{z, N, bias, nullptr, y}, st);
  }
  if (gate) return launch<T>(A, lda, W, K, M, N, K, EpiResidual<1>{z, N, bias, gate}, st);
  return launch<T>(A, lda, W, K, M, N, K, EpiResidual<0>{z, N, bias, nullptr}, st);
}

template <typename T>
hipError_t gemm_patch(const T* A, const T* W, int M, int d, int P, const float* bias, float* z,
                      hipStream_t st) {
  EpiPatch e{z, d, bias};
  return launch<T>(A, P, W, P, M, d, P, e, st);
}

template <typename T>
hipError_t gemm_head(const T* A, const T* W, int M, int d, int P, const float* bias, float* out,
                     const int* slot_id, int L, int gh, int gw, int F, int H, int Wd, long D,
                     hipStream_t st) {
  EpiHead e{out, slot_id, bias, L, gh, gw, F, H, Wd, D};
  return launch_staged<T, GemmCfgNarrow<T>>(A, d, W, d, M, P, d, e, st);
}

#define CS_INST(T)                                                                              \
  template hipError_t gemm_store<T>(const T*, long, const T*, int, int, int, const float*, int, \
                                    T*, long, hipStream_t);                                     \
  template hipError_t gemm_store_t<T>(const T*, long, const T*, int, int, int, const float*,   \
                                      T*, long, hipStream_t);                                   \
  template hipError_t gemm_qkv<T>(const T*, const T*, int, int, const float*, int, T*, T*,     \
                                  long, hipStream_t);                                           \
  template hipError_t gemm_residual<T>(const T*, long, const T*, int, int, int, const float*,  \
                                       const float*, float*, T*, hipStream_t);                  \
  template hipError_t gemm_patch<T>(const T*, const T*, int, int, int, const float*, float*,   \
                                    hipStream_t);                                               \
  template hipError_t gemm_head<T>(const T*, const T*, int, int, int, const float*, float*,    \
                                   const int*, int, int, int, int, int, int, long, hipStream_t);
CS_INST(bf16)
CS_INST(float)
#undef CS_INST

}  // namespace cs
