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

#include <type_traits>

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

// Accumulator layout of the register-staged kernel: the products are formed as C^T
// tiles (W fragment as the MFMA A operand), so accumulator (i, j) of a lane
// holds row i*32 + lane%32 of the wave's sub-tile and, in register 4g + r,
// column j*32 + 8g + 4(lane/32) + r.  Every group of 4 registers is 4
// consecutive columns of one row, i.e. one vector access in the epilogue.
//
// Every projection of the model has a bias; the accumulators start from it
// (each column's bias, then the products in a fixed K order), so the
// epilogue reads no bias.
template <int TM, int TN>
CS_DEV void init_acc_bias(f32x16 (&acc)[TM][TN], const float* __restrict__ bias, int col_base,
                          int lane, int N) {
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int col0 = col_base + j * 32 + 8 * g + 4 * (lane >> 5);
      float4 b = make_float4(0.f, 0.f, 0.f, 0.f);
      if (col0 < N) b = *reinterpret_cast<const float4*>(bias + col0);
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        acc[i][j][4 * g] = b.x;
        acc[i][j][4 * g + 1] = b.y;
        acc[i][j][4 * g + 2] = b.z;
        acc[i][j][4 * g + 3] = b.w;
      }
    }
}

// Epilogue over the wave's accumulators, in chunks of one accumulator (4
// groups of 4 columns).  The operands an epilogue reads (Epi::pre: residual
// and gate) are requested one chunk ahead of the chunk being stored, so their
// latency overlaps the previous chunk's arithmetic and stores instead of
// stalling every group.  A wave whose sub-tile lies inside [0,M) x [0,N)
// (all but the tail tiles) takes a copy without bounds checks: straight-line
// code lets the compiler wait for exactly the loads it needs, where branches
// around each access would make it wait for all outstanding memory traffic.
template <bool CHECK, int TM, int TN, class Epi>
CS_DEV void gemm_epilogue_impl(const f32x16 (&acc)[TM][TN], int row_base, int col_base, int lane,
                               int M, int N, const Epi& epi) {
  constexpr int NQ = TM * TN;
  typename Epi::Pre pre[2][4];
  auto fetch = [&](int q, int slot) {
    const int i = q / TN, j = q % TN;
    const int row = row_base + i * 32 + (lane & 31);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int col0 = col_base + j * 32 + 8 * g + 4 * (lane >> 5);
      if (!CHECK || (row < M && col0 < N)) pre[slot][g] = epi.pre(row, col0);
    }
  };
  fetch(0, 0);
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    if (q + 1 < NQ) fetch(q + 1, (q + 1) & 1);
    const int i = q / TN, j = q % TN;
    const int row = row_base + i * 32 + (lane & 31);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int col0 = col_base + j * 32 + 8 * g + 4 * (lane >> 5);
      if (!CHECK || (row < M && col0 < N)) {
        const float v[4] = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                            acc[i][j][4 * g + 3]};
        epi(row, col0, v, pre[q & 1][g]);
      }
    }
  }
}

template <int TM, int TN, class Epi>
CS_DEV void gemm_epilogue(const f32x16 (&acc)[TM][TN], int row_base, int col_base, int lane,
                          int M, int N, const Epi& epi) {
  if (row_base + TM * 32 <= M && col_base + TN * 32 <= N)
    gemm_epilogue_impl<false>(acc, row_base, col_base, lane, M, N, epi);
  else
    gemm_epilogue_impl<true>(acc, row_base, col_base, lane, M, N, epi);
}

// LDS layout of the direct-load bf16 kernels: a tile row holds 64 bf16 (8
// chunks of 16 bytes); logical chunk c of row r is stored at c ^ gemm_swz(r),
// gemm_swz(r) = r mod 8.  A fragment read (16 rows, each lane one 16-byte
// chunk) measured free of LDS bank conflicts with this swizzle (a variant
// that also flips chunk bit 0 for rows 8..15 of each 16 stalled the LDS on
// conflicts 14% of the kernel's cycles).  Rows r and r + 16 share the
// swizzle, so the fragment reads of the 16-row blocks of a wave tile differ
// by an immediate offset.
CS_DEV int gemm_swz(int r) { return r & 7; }

// 16x16 accumulators of the bf16 kernel (v_mfma_f32_16x16x32_bf16), also
// formed as C^T tiles: accumulator (i, j) of a lane holds row i*16 + lane%16
// of the wave's sub-tile and, in registers 0..3, columns j*16 + 4(lane/16) ..
// +3, one vector access in the epilogue.
template <int TM, int TN>
CS_DEV void init_acc16_bias(f32x4 (&acc)[TM][TN], const float* __restrict__ bias, int col_base,
                            int lane, int N) {
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int col0 = col_base + j * 16 + 4 * (lane >> 4);
    float4 b = make_float4(0.f, 0.f, 0.f, 0.f);
    if (col0 < N) b = *reinterpret_cast<const float4*>(bias + col0);
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      acc[i][j][0] = b.x;
      acc[i][j][1] = b.y;
      acc[i][j][2] = b.z;
      acc[i][j][3] = b.w;
    }
  }
}

// Epilogue over 16x16 accumulators, one accumulator (4 columns of one row)
// per step, the next step's epilogue operands fetched ahead.
template <bool CHECK, int TM, int TN, class Epi>
CS_DEV void gemm_epilogue16_impl(const f32x4 (&acc)[TM][TN], int row_base, int col_base, int lane,
                                 int M, int N, const Epi& epi) {
  constexpr int NQ = TM * TN;
  typename Epi::Pre pre[2];
  auto fetch = [&](int q, int slot) {
    const int i = q / TN, j = q % TN;
    const int row = row_base + i * 16 + (lane & 15);
    const int col0 = col_base + j * 16 + 4 * (lane >> 4);
    if (!CHECK || (row < M && col0 < N)) pre[slot] = epi.pre(row, col0);
  };
  fetch(0, 0);
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    if (q + 1 < NQ) fetch(q + 1, (q + 1) & 1);
    const int i = q / TN, j = q % TN;
    const int row = row_base + i * 16 + (lane & 15);
    const int col0 = col_base + j * 16 + 4 * (lane >> 4);
    if (!CHECK || (row < M && col0 < N)) {
      const float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
      epi(row, col0, v, pre[q & 1]);
    }
  }
}

template <int TM, int TN, class Epi>
CS_DEV void gemm_epilogue16(const f32x4 (&acc)[TM][TN], int row_base, int col_base, int lane, int M,
                            int N, const Epi& epi) {
  if (row_base + TM * 16 <= M && col_base + TN * 16 <= N)
    gemm_epilogue16_impl<false>(acc, row_base, col_base, lane, M, N, epi);
  else
    gemm_epilogue16_impl<true>(acc, row_base, col_base, lane, M, N, epi);
}

// OCC = waves per SIMD the register budget is sized for; GM = tile-rows per
// group of the tile order (1 = row-major).
template <typename T, int BM, int BN, int BK, int WM, int WN, int NWAVE, int OCC, int GM, class Epi>
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
  // (workgroups are dealt round-robin to the 8 dies).  Inside a range, tiles
  // are visited in groups of GM tile-rows, column-major within the group, so
  // the workgroups resident on one die at a time share both rows of A and
  // columns of W in its L2.
  const int tiles_n = (N + BN - 1) / BN;
  const int tiles_m = (M + BM - 1) / BM;
  const int nwg = gridDim.x;
  const int bid = xcd_contiguous(blockIdx.x, nwg);
  int tm_i, tn_i;
  if (GM > 1) {
    const int group = bid / (GM * tiles_n);
    const int first_m = group * GM;
    const int gm = min(tiles_m - first_m, GM);
    const int in = bid - group * GM * tiles_n;
    tm_i = first_m + in % gm;
    tn_i = in / gm;
  } else {
    tm_i = bid / tiles_n;
    tn_i = bid % tiles_n;
  }
  const int m0 = tm_i * BM;
  const int n0 = tn_i * BN;

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
  init_acc_bias(acc, epi.bias, n0 + wn * WN, lane, N);

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
        for (int j = 0; j < S::TN; ++j) acc[i][j] = MF::mma(fb[c][j], fa[c][i], acc[i][j]);
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

  gemm_epilogue(acc, m0 + wm * WM, n0 + wn * WN, lane, M, N, epi);
}

// ---------------------------------------------------------------------------
// bf16 GEMM with direct global->LDS loads (gfx950 buffer_load_dwordx4 ... lds)
// and 16x16x32 MFMAs.
//
// Each load instruction of a wave moves 64 x 16 bytes into 1 KB of LDS at
// base + 16*lane, with an arbitrary source offset per lane, so no registers
// stage the tiles and no LDS store instructions are issued.  K slices rotate
// through a ring of STAGES buffers: slice k+STAGES-1 is requested while slice
// k is multiplied, and a wave waits (vmcnt) only for slice k before the single
// barrier of each iteration (STAGES = 2: slice k+1 is requested while slice
// k is multiplied).  LDS rows are unpadded and swizzled (gemm_swz), which
// keeps the fragment reads (16 rows x 4 chunks per instruction) free of bank
// conflicts.
//
// The 16x16x32 product gives bitwise the same sums as two chained 32x32x16
// steps over the same K order (checked at all projection shapes), and measured
// 3-6% faster at the Wan2.1-1.3B projection sizes: with the same wave tile
// the fragment reads and products interleave more finely.
// ---------------------------------------------------------------------------
template <int BM, int BN, int BK, int WM, int WN, int NWAVE, int OCC, int STAGES, int GM,
          class Epi>
__global__ __launch_bounds__(64 * NWAVE, OCC) void k_gemm_dl(const bf16* __restrict__ A, long lda,
                                                           const bf16* __restrict__ W, long ldw,
                                                           int M, int N, int K, Epi epi) {
  constexpr int CH = 8;                       // bf16 per 16-byte chunk
  constexpr int CPR = BK / CH;                // chunks per LDS row
  constexpr int RPI = 64 / CPR;               // rows filled by one wave instruction
  constexpr int A_INST = BM / RPI / NWAVE;    // load instructions per wave per slice
  constexpr int B_INST = BN / RPI / NWAVE;
  constexpr int PER_SLICE = A_INST + B_INST;
  constexpr int STAGE = (BM + BN) * BK;       // elements per stage
  constexpr int WAVES_N = BN / WN;
  constexpr int TM = WM / 16, TN = WN / 16;  // 16x16 accumulators per wave
  constexpr int KS = BK / 32;                 // MFMA k-steps per slice
  static_assert(A_INST * RPI * NWAVE == BM && B_INST * RPI * NWAVE == BN, "load split");
  static_assert((BM / WM) * WAVES_N == NWAVE, "wave grid");
  static_assert(STAGES == 2, "two-stage ring");
  static_assert(KS == 2, "two k-steps per slice");
  static_assert(BN * BK * 2 == 32768 && RPI * BK * 2 == 1024, "tiled W block layout");
  __shared__ __attribute__((aligned(1024))) bf16 smem[STAGES * STAGE];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;

  const int tiles_n = (N + BN - 1) / BN;
  const int tiles_m = (M + BM - 1) / BM;
  const int nwg = gridDim.x;
  const int bid = xcd_contiguous(blockIdx.x, nwg);
  int tm_i, tn_i;
  if (GM > 1) {
    const int group = bid / (GM * tiles_n);
    const int first_m = group * GM;
    const int gm = min(tiles_m - first_m, GM);
    const int in = bid - group * GM * tiles_n;
    tm_i = first_m + in % gm;
    tn_i = in / gm;
  } else {
    tm_i = bid / tiles_n;
    tn_i = bid % tiles_n;
  }
  const int m0 = tm_i * BM, n0 = tn_i * BN;

  // per-lane sources: lane covers row (lane / CPR) of its instruction's rows
  // and physical chunk lane % CPR, i.e. logical chunk phys ^ f(row).  One
  // buffer range per operand starts at the tile's first row and covers the
  // rows that exist, so rows of a ragged last tile load as zeros.
  //
  // W is stored pre-tiled (gemm_tile_weight): the BN x BK block of tile-column
  // tn and slice kt is 32 KB contiguous at ((tn * nk + kt) * BN * BK)
  // elements, already in this kernel's LDS layout, so each load instruction
  // copies 1 KB contiguous.
  const bf16* a_base = A + (long)m0 * lda;
  const bf16* b_base = W + (long)tn_i * BN * K;
  const int a_bytes = min(BM, M - m0) * (int)lda * 2, b_bytes = BN * K * 2;
  int a_off[A_INST], b_off[B_INST];
  {
    const int rin = lane / CPR, phys = lane % CPR;
#pragma unroll
    for (int i = 0; i < A_INST; ++i) {
      const int row = (wave * A_INST + i) * RPI + rin;
      a_off[i] = (row * (int)lda + (phys ^ gemm_swz(row)) * CH) * 2;
    }
#pragma unroll
    for (int i = 0; i < B_INST; ++i) b_off[i] = (wave * B_INST + i) * 1024 + lane * 16;
  }
  auto issue = [&](int slice, int st) {
    bf16* sa = smem + st * STAGE;
    bf16* sb = sa + BM * BK;
#pragma unroll
    for (int i = 0; i < A_INST; ++i)
      buffer_load_lds16(a_base, a_bytes, sa + (wave * A_INST + i) * RPI * BK, a_off[i], slice * BK * 2);
#pragma unroll
    for (int i = 0; i < B_INST; ++i)
      buffer_load_lds16(b_base, b_bytes, sb + (wave * B_INST + i) * RPI * BK, b_off[i],
                        slice * BN * BK * 2);
  };

  f32x4 acc[TM][TN];
  init_acc16_bias(acc, epi.bias, n0 + wn * WN, lane, N);

  const int nk = K / BK;
  issue(0, 0);

  // fragment addressing (16x16x32 operands): lane reads row (lane & 15) of
  // each 16-row block at logical chunk 4*ks + (lane >> 4)
  const int a_row0 = wm * WM + (lane & 15);
  const int b_row0 = wn * WN + (lane & 15);
  const int quad = lane >> 4;

  // One slice: wait for it, request the next one into the other stage, then
  // the products of its two k-steps.  The instruction order inside a slice is
  // fixed with scheduling groups: the next slice's loads and k-step 0's
  // fragment reads first, then k-step 0's products with k-step 1's fragment
  // reads spread among them, then k-step 1's products.  The last slice is
  // peeled so that each slice is one straight-line block.
  auto slice = [&](int kt, auto more) {
    wait_vm_barrier<0>();
    if constexpr (decltype(more)::value) issue(kt + 1, (kt + 1) & 1);
    const bf16* sa = smem + (kt & 1) * STAGE;
    const bf16* sb = sa + BM * BK;
    bf16x8 fa[KS][TM], fb[KS][TN];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int c = 4 * ks + quad;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = a_row0 + i * 16;
        fa[ks][i] = *reinterpret_cast<const bf16x8*>(sa + r * BK + (c ^ gemm_swz(r)) * CH);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int r = b_row0 + j * 16;
        fb[ks][j] = *reinterpret_cast<const bf16x8*>(sb + r * BK + (c ^ gemm_swz(r)) * CH);
      }
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[ks][j], fa[ks][i], acc[i][j], 0, 0, 0);
    // NM / NF products per fragment read (rounded down: with 8 x 4
    // accumulators, 2 products per read, the rest of k-step 0 and k-step 1
    // after the reads)
    constexpr int NF = TM + TN, NM = TM * TN;
    __builtin_amdgcn_sched_group_barrier(0x020, decltype(more)::value ? PER_SLICE : 0, 0);  // VMEM
    __builtin_amdgcn_sched_group_barrier(0x100, NF, 0);                                    // DS read
#pragma unroll
    for (int i = 0; i < NF; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, NM / NF, 0);                             // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
  };
  typedef std::integral_constant<bool, true> More;
  typedef std::integral_constant<bool, false> Last;
  for (int kt = 0; kt + 1 < nk; ++kt) slice(kt, More{});
  slice(nk - 1, Last{});

  gemm_epilogue16(acc, m0 + wm * WM, n0 + wn * WN, lane, M, N, epi);
}

// Epilogue over 16x16 accumulators with the epilogue operands of PD - 1
// chunks in flight (a ring of PD slots): with one wave per SIMD nothing else
// hides the latency of the residual reads, so they are requested well ahead.
template <bool CHECK, int PD, int TM, int TN, class Epi>
CS_DEV void gemm_epilogue16_deep_impl(const f32x4 (&acc)[TM][TN], int row_base, int col_base,
                                      int lane, int M, int N, const Epi& epi) {
  constexpr int NQ = TM * TN;
  typename Epi::Pre pre[PD];
  auto fetch = [&](int q) {
    const int i = q / TN, j = q % TN;
    const int row = row_base + i * 16 + (lane & 15);
    const int col0 = col_base + j * 16 + 4 * (lane >> 4);
    if (!CHECK || (row < M && col0 < N)) pre[q % PD] = epi.pre(row, col0);
  };
#pragma unroll
  for (int q = 0; q < PD - 1 && q < NQ; ++q) fetch(q);
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    if (q + PD - 1 < NQ) fetch(q + PD - 1);
    const int i = q / TN, j = q % TN;
    const int row = row_base + i * 16 + (lane & 15);
    const int col0 = col_base + j * 16 + 4 * (lane >> 4);
    if (!CHECK || (row < M && col0 < N)) {
      const float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
      epi(row, col0, v, pre[q % PD]);
    }
  }
}

template <int PD, int TM, int TN, class Epi>
CS_DEV void gemm_epilogue16_deep(const f32x4 (&acc)[TM][TN], int row_base, int col_base, int lane,
                                 int M, int N, const Epi& epi) {
  if (row_base + TM * 16 <= M && col_base + TN * 16 <= N)
    gemm_epilogue16_deep_impl<false, PD>(acc, row_base, col_base, lane, M, N, epi);
  else
    gemm_epilogue16_deep_impl<true, PD>(acc, row_base, col_base, lane, M, N, epi);
}

// ---------------------------------------------------------------------------
// bf16 GEMM, one wave per SIMD: BM x 256 tiles (BM = 256 or 192), 4 waves of
// (BM/2) x 128 (16x16x32 MFMAs; BM/2 x 128 / 64 accumulator registers per
// lane, held in AGPRs).
//
// Fragment reads from LDS per product: (BM/32 + 8) reads per BM/4 products,
// against 12 per 32 with 8 waves of 128x64, so the LDS, which also absorbs
// the direct loads, is less of a co-limit.  With a single wave per SIMD no
// other wave hides a stall, so every LDS read is issued half a K slice (one
// k-step of products) ahead of its use, and the direct loads are spread
// evenly over the slice (clumped, they back up the address unit and stall
// the issuing wave):
//
//   slice k, half 1: products of k-step 0 | reads of k-step 1 of slice k |
//                    loads of the A rows of slice k+2
//   wait: own loads of slice k+1 landed, own reads done; barrier
//   slice k, half 2: products of k-step 1 | reads of k-step 0 of slice k+1 |
//                    loads of the W rows of slice k+2
//
// A tiles rotate through three LDS buffers and W tiles through two (160 KB
// at BM = 256): the A buffer of slice k+2 held slice k-1, which every wave
// finished reading before the previous barrier, and the W buffer of slice
// k+2 held slice k, whose last reads precede this slice's barrier.
//
// The products are issued as volatile inline assembly with the accumulators
// bound to AGPRs: that fixes the issue order exactly (LDS reads and loads
// are ordered against them) and keeps the register allocator from moving
// accumulators between the register files.  The compiler does not see them
// as matrix instructions, so the hazards it would otherwise cover are
// covered here: the accumulators are written (bias) long before the first
// product, none is read until 24 wait states after the last product, and a
// fragment register is rewritten by an LDS read no sooner than eight
// products after the last product that used it.
//
// Same LDS row layout, tiled weights, tile order and accumulation order over
// K as k_gemm_dl: results are bitwise equal to it.
// ---------------------------------------------------------------------------
// Epilogues that route a workgroup's tile through LDS on its way out
// (staged_tile / store_staged_tile), once the main loop has released the
// ring: each wave gets a region of max(WN (WM + 8), WM (WN + 8)) elements.
template <class Epi> struct EpiStagesTiles : std::false_type {};

CS_DEV void mfma_16x16x32_agpr(f32x4& acc, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}

template <int BM, int GM, int PD, class Epi>
__global__ __launch_bounds__(256, 1) void k_gemm_w4(const bf16* __restrict__ A, long lda,
                                                  const bf16* __restrict__ W, long ldw, int M,
                                                  int N, int K, Epi epi) {
  constexpr int BN = 256, BK = 64, NWAVE = 4, WM = BM / 2, WN = 128;
  constexpr int CH = 8;                       // bf16 per 16-byte chunk
  constexpr int CPR = BK / CH;                // chunks per LDS row
  constexpr int RPI = 64 / CPR;               // rows filled by one wave instruction
  constexpr int A_INST = BM / RPI / NWAVE;    // load instructions per wave per slice
  constexpr int B_INST = BN / RPI / NWAVE;
  constexpr int A_BUF = BM * BK, B_BUF = BN * BK;  // elements per buffer
  constexpr int WAVES_N = BN / WN;
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int NF = TM + TN, NM = TM * TN;   // reads and products per k-step
  constexpr int RPM = 3;                      // products per read
  static_assert(BM == 256 || BM == 192, "tile rows");
  static_assert(A_INST * RPI * NWAVE == BM && B_INST * RPI * NWAVE == BN, "load split");
  static_assert(BN * BK * 2 == 32768 && RPI * BK * 2 == 1024, "tiled W block layout");
  static_assert(RPM * (NF - 1) < NM && NM % A_INST == 0 && NM % B_INST == 0, "interleave");
  __shared__ __attribute__((aligned(1024))) bf16 smem[3 * A_BUF + 2 * B_BUF];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;

  const int tiles_n = (N + BN - 1) / BN;
  const int tiles_m = (M + BM - 1) / BM;
  const int bid = xcd_contiguous(blockIdx.x, gridDim.x);
  int tm_i, tn_i;
  if (GM > 1) {
    const int group = bid / (GM * tiles_n);
    const int first_m = group * GM;
    const int gm = min(tiles_m - first_m, GM);
    const int in = bid - group * GM * tiles_n;
    tm_i = first_m + in % gm;
    tn_i = in / gm;
  } else {
    tm_i = bid / tiles_n;
    tn_i = bid % tiles_n;
  }
  const int m0 = tm_i * BM, n0 = tn_i * BN;

  const bf16* a_base = A + (long)m0 * lda;
  const bf16* b_base = W + (long)tn_i * BN * K;
  const int a_bytes = min(BM, M - m0) * (int)lda * 2, b_bytes = BN * K * 2;
  int a_off[A_INST], b_off[B_INST];
  {
    const int rin = lane / CPR, phys = lane % CPR;
#pragma unroll
    for (int i = 0; i < A_INST; ++i) {
      const int row = (wave * A_INST + i) * RPI + rin;
      a_off[i] = (row * (int)lda + (phys ^ gemm_swz(row)) * CH) * 2;
    }
#pragma unroll
    for (int i = 0; i < B_INST; ++i) b_off[i] = (wave * B_INST + i) * 1024 + lane * 16;
  }
  bf16* const sb0 = smem + 3 * A_BUF;
  // load instruction r of the A (W) rows of slice `slice` into A buffer ab (W buffer bb)
  auto load_a = [&](int r, int slice, int ab) {
    buffer_load_lds16(a_base, a_bytes, smem + ab * A_BUF + (wave * A_INST + r) * RPI * BK, a_off[r],
                      slice * BK * 2);
  };
  auto load_b = [&](int r, int slice, int bb) {
    buffer_load_lds16(b_base, b_bytes, sb0 + bb * B_BUF + (wave * B_INST + r) * RPI * BK, b_off[r],
                      slice * BN * BK * 2);
  };

  f32x4 acc[TM][TN];
  init_acc16_bias(acc, epi.bias, n0 + wn * WN, lane, N);
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) asm volatile("" : "+a"(acc[i][j]));  // in AGPRs from here on

  // fragment addressing (16x16x32 operands): lane reads row (lane & 15) of
  // each 16-row block at logical chunk 4*ks + (lane >> 4); the swizzle of
  // row r + 16i equals that of row r, so block i is at an immediate offset
  const int a_row0 = wm * WM + (lane & 15);
  const int b_row0 = wn * WN + (lane & 15);
  const int quad = lane >> 4;
  const int a_lds[2] = {a_row0 * BK + (quad ^ gemm_swz(a_row0)) * CH,
                        a_row0 * BK + ((4 + quad) ^ gemm_swz(a_row0)) * CH};
  const int b_lds[2] = {b_row0 * BK + (quad ^ gemm_swz(b_row0)) * CH,
                        b_row0 * BK + ((4 + quad) ^ gemm_swz(b_row0)) * CH};
  // read r (< NF) of k-step ks from A buffer ab / W buffer bb: W fragments
  // first (the first products of the next half use all of them)
  auto read = [&](int r, int ab, int bb, int ks, bf16x8(&fa)[TM], bf16x8(&fb)[TN]) {
    if (r < TN)
      fb[r] = *reinterpret_cast<const bf16x8*>(sb0 + bb * B_BUF + b_lds[ks] + r * 16 * BK);
    else
      fa[r - TN] = *reinterpret_cast<const bf16x8*>(smem + ab * A_BUF + a_lds[ks] + (r - TN) * 16 * BK);
  };

  bf16x8 f0a[TM], f0b[TN], f1a[TM], f1b[TN];
  // One half: the NM products of (pa, pb); after product RPM*r, read r into
  // (na, nb) (RD); NL loads spread evenly, through `ld` (LD).
  auto half = [&](auto rd, auto ldf, auto nl, const bf16x8(&pa)[TM], const bf16x8(&pb)[TN],
                  bf16x8(&na)[TM], bf16x8(&nb)[TN], int ab, int bb, int ks) {
    constexpr int NL = decltype(nl)::value;
#pragma unroll
    for (int q = 0; q < NM; ++q) {
      mfma_16x16x32_agpr(acc[q / TN][q % TN], pb[q % TN], pa[q / TN]);
      if constexpr (NL > 0) {
        if (q % (NM / NL) == NM / NL / 2) ldf(q / (NM / NL));
      }
      if constexpr (decltype(rd)::value) {
        if (q % RPM == 0 && q / RPM < NF) read(q / RPM, ab, bb, ks, na, nb);
      }
    }
  };
  typedef std::integral_constant<bool, true> Y;
  typedef std::integral_constant<bool, false> F;
  typedef std::integral_constant<int, 0> L0;
  typedef std::integral_constant<int, A_INST> LA;
  typedef std::integral_constant<int, B_INST> LB;
  auto no_load = [](int) {};

  const int nk = K / BK;
#pragma unroll
  for (int r = 0; r < A_INST; ++r) load_a(r, 0, 0);
#pragma unroll
  for (int r = 0; r < B_INST; ++r) load_b(r, 0, 0);
  if (nk > 1) {
#pragma unroll
    for (int r = 0; r < A_INST; ++r) load_a(r, 1, 1);
#pragma unroll
    for (int r = 0; r < B_INST; ++r) load_b(r, 1, 1);
    wait_vm_barrier<A_INST + B_INST>();   // slice 0 landed (slice 1 may be in flight)
  } else {
    wait_vm_barrier<0>();
  }
#pragma unroll
  for (int r = 0; r < NF; ++r) read(r, 0, 0, 0, f0a, f0b);

  // HN: slice k+1 exists (barrier, its k-step 0 reads); IS: slice k+2
  // exists (its loads).  Slice k uses A buffer k % 3 and W buffer k % 2.
  auto slice = [&](int kt, int a3, auto hn, auto is) {
    const int b2 = kt & 1;
    const int a_next = a3 == 2 ? 0 : a3 + 1, a_far = a3 == 0 ? 2 : a3 - 1;
    if constexpr (decltype(is)::value) {
      half(Y{}, [&](int r) { load_a(r, kt + 2, a_far); }, LA{}, f0a, f0b, f1a, f1b, a3, b2, 1);
      asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(A_INST) : "memory");
      half(Y{}, [&](int r) { load_b(r, kt + 2, b2); }, LB{}, f1a, f1b, f0a, f0b, a_next, b2 ^ 1, 0);
    } else if constexpr (decltype(hn)::value) {
      half(Y{}, no_load, L0{}, f0a, f0b, f1a, f1b, a3, b2, 1);
      asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
      half(Y{}, no_load, L0{}, f1a, f1b, f0a, f0b, a_next, b2 ^ 1, 0);
    } else {
      half(Y{}, no_load, L0{}, f0a, f0b, f1a, f1b, a3, b2, 1);
      half(F{}, no_load, L0{}, f1a, f1b, f0a, f0b, 0, 0, 0);
    }
  };
  int kt = 0, a3 = 0;
  for (; kt + 2 < nk; ++kt, a3 = a3 == 2 ? 0 : a3 + 1) slice(kt, a3, Y{}, Y{});
  if (kt + 1 < nk) {
    slice(kt, a3, Y{}, F{});
    ++kt;
    a3 = a3 == 2 ? 0 : a3 + 1;
  }
  slice(kt, a3, F{}, F{});

  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7");
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) asm volatile("" : "+a"(acc[i][j]));  // read only after the nops
  if constexpr (EpiStagesTiles<Epi>::value) {
    constexpr int STG = WN * (WM + 8) > WM * (WN + 8) ? WN * (WM + 8) : WM * (WN + 8);
    static_assert(NWAVE * STG <= 3 * A_BUF + 2 * B_BUF, "staging fits the ring");
    if (epi.staged_tile(n0)) {   // uniform over the workgroup
      __syncthreads();           // every wave's last fragment reads are done
      epi.store_staged_tile(acc, smem + wave * STG, m0 + wm * WM, n0 + wn * WN, lane, M, N);
      return;
    }
  }
  gemm_epilogue16_deep<PD>(acc, m0 + wm * WM, n0 + wn * WN, lane, M, N, epi);
}

// ------------------------------------------------------------- epilogues
// Each epilogue is called per (row, 4 consecutive columns col0..col0+3) with
// the accumulated values v (bias included); N is a multiple of 4.  `Pre` is
// what it reads from memory besides v, fetched ahead by `pre`.
template <typename T> CS_DEV void store4(T* p, const float* y) {
  if constexpr (sizeof(T) == 2) {
    bf16x4 q;
#pragma unroll
    for (int r = 0; r < 4; ++r) q[r] = to_t<T>(y[r]);
    *reinterpret_cast<bf16x4*>(p) = q;
  } else {
    *reinterpret_cast<float4*>(p) = make_float4(y[0], y[1], y[2], y[3]);
  }
}
struct NoPre {};

// Row-major bf16 store of one wave's TM*16 x TN*16 block of 16x16
// accumulators (lane holds row row_base + 16i + (lane & 15), columns
// col_base + 16j + 4(lane >> 4) + r) through `stage` (TM*16 rows of TN*16 + 8
// elements): written as 8-byte pieces, read back and stored as 16-byte runs,
// 256 contiguous bytes per row, where the direct path stores 32-byte pieces
// of 16 rows per instruction.  f maps each value before its rounding.
// Contains one workgroup barrier: every wave of the workgroup calls a staged
// store exactly once.
template <int TM, int TN, class F>
CS_DEV void store_rows_staged(const f32x4 (&acc)[TM][TN], bf16* stage, int row_base, int col_base,
                              int lane, int M, int N, bf16* out, long ldo, F f) {
  constexpr int R = TM * 16, C = TN * 16, SP = C + 8;
  constexpr int LPR = C / 8, RPI = 64 / LPR;   // lanes per row, rows per instruction
  static_assert(64 % LPR == 0 && R % RPI == 0, "readback split");
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      bf16x4 q;
#pragma unroll
      for (int r = 0; r < 4; ++r) q[r] = (bf16)f(acc[i][j][r]);
      *reinterpret_cast<bf16x4*>(stage + (16 * i + (lane & 15)) * SP + 16 * j + 4 * (lane >> 4)) = q;
    }
  __syncthreads();
  const int c = 8 * (lane % LPR), col = col_base + c;
  const bool whole = col + 8 <= N && ((ldo | col) & 7) == 0;
#pragma unroll 4
  for (int q = 0; q < R / RPI; ++q) {
    const int r = RPI * q + lane / LPR, row = row_base + r;
    if (row >= M) continue;
    const bf16x8 v = *reinterpret_cast<const bf16x8*>(stage + r * SP + c);
    bf16* dst = out + (long)row * ldo + col;
    if (whole && ((uintptr_t)dst & 15) == 0) {
      *reinterpret_cast<bf16x8*>(dst) = v;
    } else {
      for (int e = 0; e < 8 && col + e < N; ++e) dst[e] = v[e];
    }
  }
}

struct IdentityF { CS_DEV float operator()(float x) const { return x; } };
struct GeluF { CS_DEV float operator()(float x) const { return gelu_tanh(x); } };

// On the bf16 kernel every tile goes out through LDS (store_rows_staged).
// Measured against the element-wise path at 8 x 32,760 rows, d = 1536, same
// process: cross q (N = 1536) 1.036 -> 0.938 ms, q|k (N = 3072) 2.032 ->
// 1.895 ms, FFN up + GELU (N = 8960) unchanged (5.877 vs 5.886 ms); same
// values.
template <typename T, int ACT> struct EpiStore {  // ACT: 0 none, 1 tanh-GELU
  T* out; long ldo; const float* bias;
  typedef NoPre Pre;
  CS_DEV Pre pre(int, int) const { return {}; }
  CS_DEV void operator()(int row, int col0, const float* v, const Pre&) const {
    float y[4] = {v[0], v[1], v[2], v[3]};
    if constexpr (ACT == 1) {
#pragma unroll
      for (int r = 0; r < 4; ++r) y[r] = gelu_tanh(y[r]);
    }
    store4<T>(out + (long)row * ldo + col0, y);
  }

  CS_DEV bool staged_tile(int) const { return true; }
  template <int TM, int TN>
  CS_DEV void store_staged_tile(const f32x4 (&acc)[TM][TN], bf16* stage, int row_base, int col_base,
                                int lane, int M, int N) const {
    static_assert(sizeof(T) == 2, "bf16 tiles only");
    if constexpr (ACT == 1)
      store_rows_staged(acc, stage, row_base, col_base, lane, M, N, out, ldo, GeluF{});
    else
      store_rows_staged(acc, stage, row_base, col_base, lane, M, N, out, ldo, IdentityF{});
  }
};
template <int ACT> struct EpiStagesTiles<EpiStore<bf16, ACT>> : std::true_type {};

// Self-attention projection: columns [0, 2d) are q and k, stored row-major
// [row][2d]; columns [2d, 3d) are v, stored transposed per stream as
// vT[stream][channel][token] with a padded token stride.
//
// On the bf16 kernel every tile goes out through LDS.  A wave whose 128
// columns lie in v (2d is a multiple of 128) writes its 128 x 128 block there
// as [channel][token] (token stride 136, 16-byte aligned rows) and stores it
// back as 16-byte runs of 8 tokens, 256 contiguous bytes per channel, where
// the element-wise path below issues a 2-byte store per value (measured: the
// v part alone: 3.386 -> 3.167 ms for the QKV projection at 8 x 32,760 rows,
// d = 1536, within 0.5% of storing v row-major); a wave in q|k stores its
// rows through store_rows_staged (both parts staged: 3.203 -> 2.886 ms;
// bitwise equal).
template <typename T> struct EpiQKV {
  T* qk; T* vt; const float* bias; int d; int L; long vt_ld; long vt_ss;
  typedef NoPre Pre;
  CS_DEV Pre pre(int, int) const { return {}; }
  CS_DEV void operator()(int row, int col0, const float* v, const Pre&) const {
    if (col0 < 2 * d) {
      store4<T>(qk + (long)row * (2 * d) + col0, v);
    } else {
      const int s = row / L, tok = row - s * L;
      T* dst = vt + (long)s * vt_ss + (long)(col0 - 2 * d) * vt_ld + tok;
#pragma unroll
      for (int r = 0; r < 4; ++r) dst[(long)r * vt_ld] = to_t<T>(v[r]);
    }
  }

  CS_DEV bool staged_tile(int) const { return true; }

  template <int TM, int TN>
  CS_DEV void store_staged_tile(const f32x4 (&acc)[TM][TN], bf16* stage, int row_base, int col_base,
                                int lane, int M, int N) const {
    static_assert(sizeof(T) == 2, "bf16 tiles only");
    if (col_base >= 2 * d)
      store_v_transposed(acc, stage, row_base, col_base, lane, M, N);
    else
      store_rows_staged(acc, stage, row_base, col_base, lane, M, 2 * d, qk, 2L * d, IdentityF{});
  }

  // One wave's TM*16 x TN*16 block of 16x16 accumulators (lane holds row
  // row_base + 16i + (lane & 15), columns col_base + 16j + 4(lane >> 4) + r)
  // through `stage` (TN*16 rows of TM*16 + 8 tokens) to vT; one workgroup
  // barrier, like store_rows_staged.
  template <int TM, int TN>
  CS_DEV void store_v_transposed(const f32x4 (&acc)[TM][TN], bf16* stage, int row_base,
                                 int col_base, int lane, int M, int N) const {
    constexpr int R = TM * 16, C = TN * 16, SP = R + 8, CHUNKS = R / 8;
    static_assert(64 % CHUNKS == 0 && C % (64 / CHUNKS) == 0, "readback split");
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          stage[(16 * j + 4 * (lane >> 4) + r) * SP + 16 * i + (lane & 15)] = to_t<T>(acc[i][j][r]);
    __syncthreads();
    // lane: tokens row0..row0+7 of channels c = CPI*q + lane / CHUNKS
    constexpr int CPI = 64 / CHUNKS;
    const int k = lane % CHUNKS;
    const int row0 = row_base + 8 * k;
    const int s = row0 / L, tok = row0 - s * L;
    const bool whole = row0 + 8 <= M && tok + 8 <= L;   // one stream, all rows valid
    T* const base = vt + (long)s * vt_ss + tok;
#pragma unroll 4
    for (int q = 0; q < C / CPI; ++q) {
      const int c = CPI * q + lane / CHUNKS;
      const int col = col_base + c;
      if (col >= N) continue;
      const bf16x8 v = *reinterpret_cast<const bf16x8*>(stage + c * SP + 8 * k);
      T* dst = base + (long)(col - 2 * d) * vt_ld;
      if (whole && ((uintptr_t)dst & 15) == 0) {
        *reinterpret_cast<bf16x8*>(dst) = v;
      } else {
        for (int e = 0; e < 8; ++e) {
          const int row = row0 + e;
          if (row >= M) break;
          const int se = row / L;
          vt[(long)se * vt_ss + (long)(col - 2 * d) * vt_ld + (row - se * L)] = v[e];
        }
      }
    }
  }
};
template <> struct EpiStagesTiles<EpiQKV<bf16>> : std::true_type {};

// Transposed store of a single-stream projection: out[col][row].
template <typename T> struct EpiStoreT {
  T* out; long ldo; const float* bias;
  typedef NoPre Pre;
  CS_DEV Pre pre(int, int) const { return {}; }
  CS_DEV void operator()(int row, int col0, const float* v, const Pre&) const {
#pragma unroll
    for (int r = 0; r < 4; ++r) out[(long)(col0 + r) * ldo + row] = to_t<T>(v[r]);
  }
};

// Residual update z += gate * (acc + bias) (GATED = 0: gate 1).  The
// updated residual is stored non-temporally: it is read again only by the
// next row pass, so it need not displace the operand tiles the GEMM keeps in
// L2 (measured +2.6% on the K = 8960 projection, neutral at K = 1536).
typedef float f32x4v __attribute__((ext_vector_type(4)));
template <int GATED> struct EpiResidual {
  float* z; long ldz; const float* bias; const float* gate;
  struct Pre { float4 z, g; };
  CS_DEV Pre pre(int row, int col0) const {
    Pre p;
    p.z = *reinterpret_cast<const float4*>(z + (long)row * ldz + col0);
    p.g = make_float4(1.f, 1.f, 1.f, 1.f);
    if constexpr (GATED) p.g = *reinterpret_cast<const float4*>(gate + col0);
    return p;
  }
  CS_DEV void operator()(int row, int col0, const float* v, const Pre& p) const {
    float4 o = p.z;
    o.x += p.g.x * v[0];
    o.y += p.g.y * v[1];
    o.z += p.g.z * v[2];
    o.w += p.g.w * v[3];
    const f32x4v ov = {o.x, o.y, o.z, o.w};
    __builtin_nontemporal_store(ov, reinterpret_cast<f32x4v*>(z + (long)row * ldz + col0));
  }
};

// Residual update that also keeps the branch output y = acc + bias in y
// (row stride N, compute type) for later reuse: z += gate * y.
template <int GATED, typename T> struct EpiResidualStore {
  float* z; long ldz; const float* bias; const float* gate; T* y;
  typedef typename EpiResidual<GATED>::Pre Pre;
  CS_DEV Pre pre(int row, int col0) const {
    return EpiResidual<GATED>{z, ldz, bias, gate}.pre(row, col0);
  }
  CS_DEV void operator()(int row, int col0, const float* v, const Pre& p) const {
    store4<T>(y + (long)row * ldz + col0, v);
    EpiResidual<GATED>{z, ldz, bias, gate}(row, col0, v, p);
  }
};

// Patch embedding: z = acc + bias (fp32 residual stream).
struct EpiPatch {
  float* z; long ldz; const float* bias;
  typedef NoPre Pre;
  CS_DEV Pre pre(int, int) const { return {}; }
  CS_DEV void operator()(int row, int col0, const float* v, const Pre&) const {
    *reinterpret_cast<float4*>(z + (long)row * ldz + col0) = make_float4(v[0], v[1], v[2], v[3]);
  }
};

// Head: acc + bias, scattered back to latent layout (unpatchify).  Row
// = slot * L + token (token = (f, h, w) row-major on the patch grid);
// columns c*4 .. c*4+3 are the 2x2 patch (dy, dx) of channel c.  The slot's
// output latent is out + slot_id[slot] * D.
struct EpiHead {
  float* out; const int* slot_id; const float* bias; int L, gh, gw, F, H, Wd; long D;
  struct Pre { int slot; };
  CS_DEV Pre pre(int row, int) const { return {slot_id[row / L]}; }
  CS_DEV void operator()(int row, int col0, const float* v, const Pre& p) const {
    const int c = col0 >> 2;
    const int tok = row % L;
    const int f = tok / (gh * gw), rem = tok - f * gh * gw;
    const int hh = rem / gw, ww = rem - hh * gw;
    float* dst = out + (long)p.slot * D + (((long)c * F + f) * H + 2 * hh) * Wd + 2 * ww;
    *reinterpret_cast<float2*>(dst) = make_float2(v[0], v[1]);
    *reinterpret_cast<float2*>(dst + Wd) = make_float2(v[2], v[3]);
  }
};

}  // namespace cs
