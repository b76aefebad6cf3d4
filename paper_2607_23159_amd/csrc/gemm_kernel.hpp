// MFMA GEMM for gfx950 with fused epilogues.
//
//   C[M][N] = A[M][K] * W[N][K]^T   (A row-major, W = weights [out][in])
//
// One workgroup (4 waves) computes a BM x BN tile; each wave owns a WM x WN
// sub-tile made of 32x32 MFMA accumulators.  K is walked in BK slices that
// are staged through LDS (double buffered, one barrier per slice; the next
// slice's global loads are in flight while the current slice is multiplied).
// Rows of the LDS tiles are padded by 16 bytes so that the 16-byte fragment
// reads of 32 consecutive rows fall in distinct banks.  Ragged M and N tails
// are handled by clamping the load row (valid memory) and masking stores.
//
// The accumulation order over K is fixed by the tile shape, which depends
// only on the element type, never on M: a row's result is bitwise the same
// whatever other rows share the launch (batch invariance).
#pragma once
#include "kernels.hpp"

namespace cs {

template <typename T, int BM, int BN, int BK, int WM, int WN, int NWAVE>
struct GemmShape {
  static constexpr int NT = 64 * NWAVE;            // threads per workgroup
  static constexpr int CH = 16 / (int)sizeof(T);   // elements per 16-byte chunk
  static constexpr int LDS_LD = BK + CH;           // padded LDS row
  static constexpr int WAVES_N = BN / WN;
  static constexpr int WAVES_M = BM / WM;
  static constexpr int TM = WM / 32;
  static constexpr int TN = WN / 32;
  static constexpr int CPR = BK / CH;              // chunks per row of a slice
  static constexpr int A_CH = BM * CPR / NT;       // chunks per thread
  static constexpr int B_CH = BN * CPR / NT;
  static constexpr int KS = BK / Mfma32<T>::KSTEP; // MFMA k-steps per slice
  static_assert(WAVES_N * WAVES_M == NWAVE, "wave grid");
  static_assert(A_CH * NT == BM * CPR && B_CH * NT == BN * CPR, "slice split");
};

// OCC = waves per SIMD the register budget is sized for.
template <typename T, int BM, int BN, int BK, int WM, int WN, int NWAVE, int OCC, class Epi>
__global__ __launch_bounds__(64 * NWAVE, OCC) void k_gemm(const T* __restrict__ A, long lda,
                                                        const T* __restrict__ W, long ldw, int M,
                                                        int N, int K, Epi epi) {
  typedef GemmShape<T, BM, BN, BK, WM, WN, NWAVE> S;
  typedef Mfma32<T> MF;
  constexpr int KPL = MF::KPL, KSTEP = MF::KSTEP;
  __shared__ __attribute__((aligned(16))) T sA[2][BM * S::LDS_LD];
  __shared__ __attribute__((aligned(16))) T sB[2][BN * S::LDS_LD];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / S::WAVES_N, wn = wave % S::WAVES_N;

  // Tile order: the launch is split into 8 contiguous ranges, one per XCD
  // (workgroups are dealt round-robin to the 8 dies), so tiles that share
  // rows of A run on the same die and share its L2.
  const int tiles_n = (N + BN - 1) / BN;
  const int nwg = gridDim.x;
  int bid = blockIdx.x;
  if ((nwg & 7) == 0) bid = (bid & 7) * (nwg >> 3) + (bid >> 3);
  const int m0 = (bid / tiles_n) * BM;
  const int n0 = (bid % tiles_n) * BN;

  // global -> register staging
  Chunk16 ra[S::A_CH], rb[S::B_CH];
  const T* a_src[S::A_CH];
  const T* b_src[S::B_CH];
  int a_dst[S::A_CH], b_dst[S::B_CH];
#pragma unroll
  for (int c = 0; c < S::A_CH; ++c) {
    int id = c * S::NT + tid;
    int r = id / S::CPR, cc = id % S::CPR;
    int gr = min(m0 + r, M - 1);
    a_src[c] = A + (long)gr * lda + cc * S::CH;
    a_dst[c] = r * S::LDS_LD + cc * S::CH;
  }
#pragma unroll
  for (int c = 0; c < S::B_CH; ++c) {
    int id = c * S::NT + tid;
    int r = id / S::CPR, cc = id % S::CPR;
    int gr = min(n0 + r, N - 1);
    b_src[c] = W + (long)gr * ldw + cc * S::CH;
    b_dst[c] = r * S::LDS_LD + cc * S::CH;
  }

  f32x16 acc[S::TM][S::TN];
#pragma unroll
  for (int i = 0; i < S::TM; ++i)
#pragma unroll
    for (int j = 0; j < S::TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nk = K / BK;
#pragma unroll
  for (int c = 0; c < S::A_CH; ++c) ra[c] = ld16(a_src[c]);
#pragma unroll
  for (int c = 0; c < S::B_CH; ++c) rb[c] = ld16(b_src[c]);
#pragma unroll
  for (int c = 0; c < S::A_CH; ++c) st16(&sA[0][a_dst[c]], ra[c]);
#pragma unroll
  for (int c = 0; c < S::B_CH; ++c) st16(&sB[0][b_dst[c]], rb[c]);
  __syncthreads();

  const int frag_k = KPL * (lane >> 5);
  const int a_row = wm * WM + (lane & 31);
  const int b_row = wn * WN + (lane & 31);

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      const long koff = (long)(kt + 1) * BK;
#pragma unroll
      for (int c = 0; c < S::A_CH; ++c) ra[c] = ld16(a_src[c] + koff);
#pragma unroll
      for (int c = 0; c < S::B_CH; ++c) rb[c] = ld16(b_src[c] + koff);
    }
    const T* pa = &sA[cur][a_row * S::LDS_LD + frag_k];
    const T* pb = &sB[cur][b_row * S::LDS_LD + frag_k];
    // fragments of k-step ks+1 are read while the products of ks issue
    typename MF::frag fa[2][S::TM], fb[2][S::TN];
#pragma unroll
    for (int i = 0; i < S::TM; ++i) fa[0][i] = MF::load(pa + i * 32 * S::LDS_LD);
#pragma unroll
    for (int j = 0; j < S::TN; ++j) fb[0][j] = MF::load(pb + j * 32 * S::LDS_LD);
#pragma unroll
    for (int ks = 0; ks < S::KS; ++ks) {
      const int c = ks & 1, n = c ^ 1;
      if (ks + 1 < S::KS) {
#pragma unroll
        for (int i = 0; i < S::TM; ++i) fa[n][i] = MF::load(pa + i * 32 * S::LDS_LD + (ks + 1) * KSTEP);
#pragma unroll
        for (int j = 0; j < S::TN; ++j) fb[n][j] = MF::load(pb + j * 32 * S::LDS_LD + (ks + 1) * KSTEP);
      }
#pragma unroll
      for (int i = 0; i < S::TM; ++i)
#pragma unroll
        for (int j = 0; j < S::TN; ++j) acc[i][j] = MF::mma(fa[c][i], fb[c][j], acc[i][j]);
    }
    if (more) {
      const int nxt = cur ^ 1;
#pragma unroll
      for (int c = 0; c < S::A_CH; ++c) st16(&sA[nxt][a_dst[c]], ra[c]);
#pragma unroll
      for (int c = 0; c < S::B_CH; ++c) st16(&sB[nxt][b_dst[c]], rb[c]);
    }
    __syncthreads();
  }

  // epilogue: each lane owns, per accumulator, 4 groups of 4 consecutive rows
  // of one column.
#pragma unroll
  for (int i = 0; i < S::TM; ++i)
#pragma unroll
    for (int j = 0; j < S::TN; ++j) {
      const int col = n0 + wn * WN + j * 32 + (lane & 31);
      if (col >= N) continue;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int row0 = m0 + wm * WM + i * 32 + 8 * g + 4 * (lane >> 5);
        float v[4] = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                      acc[i][j][4 * g + 3]};
        epi(row0, col, v, M);
      }
    }
}

// ------------------------------------------------------------- epilogues
template <typename T> struct EpiStore {
  T* out; long ldo; const float* bias; int act;  // act: 0 none, 1 tanh-GELU
  CS_DEV void operator()(int row0, int col, const float* v, int M) const {
    const float b = bias ? bias[col] : 0.0f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      if (row0 + r < M) {
        float y = v[r] + b;
        if (act == 1) y = gelu_tanh(y);
        out[(long)(row0 + r) * ldo + col] = to_t<T>(y);
      }
    }
  }
};

// Self-attention projection: columns [0, 2d) are q and k, stored row-major
// [row][2d]; columns [2d, 3d) are v, stored transposed per stream as
// vT[stream][channel][token] with a padded token stride.
template <typename T> struct EpiQKV {
  T* qk; T* vt; const float* bias; int d; int L; long vt_ld; long vt_ss;
  CS_DEV void operator()(int row0, int col, const float* v, int M) const {
    const float b = bias[col];
    if (col < 2 * d) {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (row0 + r < M) qk[(long)(row0 + r) * (2 * d) + col] = to_t<T>(v[r] + b);
    } else {
      const int c = col - 2 * d;
      if ((L & 3) == 0 && row0 + 3 < M) {
        // four consecutive tokens of one stream: one 8-byte store
        const int s = row0 / L, tok = row0 - s * L;
        T* dst = vt + (long)s * vt_ss + (long)c * vt_ld + tok;
        if constexpr (sizeof(T) == 2) {
          bf16x4 q;
#pragma unroll
          for (int r = 0; r < 4; ++r) q[r] = to_t<T>(v[r] + b);
          *reinterpret_cast<bf16x4*>(dst) = q;
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) dst[r] = v[r] + b;
        }
        return;
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = row0 + r;
        if (row < M) {
          const int s = row / L, tok = row - s * L;
          vt[(long)s * vt_ss + (long)c * vt_ld + tok] = to_t<T>(v[r] + b);
        }
      }
    }
  }
};

// Transposed store of a single-stream projection: out[col][row].
template <typename T> struct EpiStoreT {
  T* out; long ldo; const float* bias;
  CS_DEV void operator()(int row0, int col, const float* v, int M) const {
    const float b = bias[col];
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (row0 + r < M) out[(long)col * ldo + row0 + r] = to_t<T>(v[r] + b);
  }
};

// Residual update z += gate * (acc + bias) (gate NULL: 1).
struct EpiResidual {
  float* z; long ldz; const float* bias; const float* gate;
  CS_DEV void operator()(int row0, int col, const float* v, int M) const {
    const float b = bias[col];
    const float g = gate ? gate[col] : 1.0f;
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (row0 + r < M) {
        float* p = z + (long)(row0 + r) * ldz + col;
        *p = *p + g * (v[r] + b);
      }
  }
};

// Patch embedding: z = acc + bias (fp32 residual stream).
struct EpiPatch {
  float* z; long ldz; const float* bias;
  CS_DEV void operator()(int row0, int col, const float* v, int M) const {
    const float b = bias[col];
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (row0 + r < M) z[(long)(row0 + r) * ldz + col] = v[r] + b;
  }
};

// Head: acc + bias, scattered back to latent layout (unpatchify).  Row
// = slot * L + token (token = (f, h, w) row-major on the patch grid);
// column = c*4 + dy*2 + dx.  The slot's output latent is out + slot_id[slot]*D.
struct EpiHead {
  float* out; const int* slot_id; const float* bias; int L, gh, gw, F, H, Wd; long D;
  CS_DEV void operator()(int row0, int col, const float* v, int M) const {
    const float b = bias[col];
    const int c = col >> 2, dy = (col >> 1) & 1, dx = col & 1;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = row0 + r;
      if (row < M) {
        const int s = row / L, tok = row - s * L;
        const int f = tok / (gh * gw), rem = tok - f * gh * gw;
        const int hh = rem / gw, ww = rem - hh * gw;
        float* dst = out + (long)slot_id[s] * D;
        dst[(((long)c * F + f) * H + 2 * hh + dy) * Wd + 2 * ww + dx] = v[r] + b;
      }
    }
  }
};

}  // namespace cs
