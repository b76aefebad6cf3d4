// Flash attention for gfx950: softmax(q k^T / sqrt(dh)) v per (stream, head),
// non-causal, online softmax in fp32, MFMA for both products.
//
// Work split.  A workgroup of NW waves shares each K/V tile; each wave owns
// QB blocks of 32 queries.  With 8 waves of one 32-query block, a wave needs
// about 200 registers, so two waves fit per SIMD and the hardware overlaps
// one wave's softmax (VALU) with the other's matrix products.
//
// Orientation.  Each wave computes the
// transposed scores S^T = K Q^T (A = K tile from LDS, B = Q^T held in
// registers for the whole key loop), so that after the softmax the
// probabilities P^T already sit in the B-operand layout of the second
// product O^T = V^T P^T (A = V^T tile from LDS).  The MFMA's contraction
// index may visit keys in any order as long as both operands agree: the
// accumulator register j of lane l holds key 8(j/4) + 4(l/32) + j%4 of a
// 32-key block, so the V^T tile is written to LDS with each 32-key block
// permuted to position 16(l/32) + j.  No shuffle of P through LDS is needed.
//
// The softmax row of query q lives in lanes l and l^32 (16 keys each per
// 32-key block), so row maxima and sums need one cross-lane exchange.
//
// K and V^T tiles of KVT keys are staged through LDS, double buffered (the
// next tile's global loads are in flight during the current tile's math).
// Keys past lk are masked to -inf in the last tile; K rows past lk are read
// clamped and V^T columns past lk must be finite (the runtime zero-fills the
// padding of every V^T buffer).
#pragma once
#include "kernels.hpp"

namespace cs {

constexpr float RESCALE_LOG2 = 8.0f;

// OCC is the number of waves per SIMD the register budget is sized for.
// CROSS distinguishes the cross-attention instantiation (text keys) from the
// self-attention one, so that profiles report them separately.
template <typename T, int DH, int QB, int KVT, int NW, int OCC, bool CROSS>
__global__ __launch_bounds__(64 * NW, OCC) void k_flash(AttnArgs<T> a) {
  typedef Mfma32<T> MF;
  constexpr int KPL = MF::KPL, KSTEP = MF::KSTEP;
  constexpr int CH = 16 / (int)sizeof(T);
  constexpr int KLD = DH + CH;    // padded K row (16 bytes)
  constexpr int VLD = KVT + CH;   // padded V^T row
  constexpr int NKT = KVT / 32;   // 32-key blocks per tile
  constexpr int NDT = DH / 32;    // 32-channel blocks of the output
  constexpr int NKS = DH / KSTEP; // k-steps of the score product
  constexpr int NPS = 32 / KSTEP; // k-steps of the value product per key block
  constexpr int NT = 64 * NW;     // threads per workgroup
  constexpr int K_CH = KVT * DH / CH / NT;
  constexpr int V_CH = DH * KVT / CH / NT;
  static_assert(K_CH * CH * NT == KVT * DH && V_CH * CH * NT == DH * KVT, "tile split");
  static_assert(CH % 4 == 0, "4-element groups");

  __shared__ __attribute__((aligned(16))) T sK[2][KVT * KLD];
  __shared__ __attribute__((aligned(16))) T sV[2][DH * VLD];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  // One flat grid over (query tile, head, stream), query tile fastest,
  // taken XCD-contiguous: the workgroups resident on one XCD at a time work
  // on the same head and read its K/V tiles through a shared L2.
  const int n_qt = (a.lq + NW * QB * 32 - 1) / (NW * QB * 32);
  const int vid = xcd_contiguous(blockIdx.x, gridDim.x);
  const int qt = vid % n_qt, hs = vid / n_qt;
  const int head = hs % a.heads, s = hs / a.heads;
  const int kvs = a.kv_sel ? a.kv_sel[s] : s;
  const int q0 = qt * (NW * QB * 32) + wave * QB * 32;

  const T* qb_ = a.q + (long)s * a.q_ss + head * DH;
  const T* kb_ = a.k + (long)kvs * a.k_ss + head * DH;
  const T* vb_ = a.vt + (long)kvs * a.vt_ss + (long)head * DH * a.vt_ld;

  // Q^T fragments (B operand), kept for the whole key loop.
  typename MF::frag qf[QB][NKS];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int row = min(q0 + qb * 32 + l32, a.lq - 1);
    const T* src = qb_ + (long)row * a.q_ld + KPL * half;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      qf[qb][ks] = MF::load(src + ks * KSTEP);
      // opaque to the optimiser: keeps Q in registers instead of reloading
      // it from memory inside the key loop
      asm volatile("" : "+v"(qf[qb][ks]));
    }
  }

  // tile staging
  Chunk16 rk[K_CH], rv[V_CH];
  auto load_tile = [&](int kv0) {
#pragma unroll
    for (int c = 0; c < K_CH; ++c) {
      const int id = c * NT + tid;
      const int r = id / (DH / CH), cc = id % (DH / CH);
      const int key = min(kv0 + r, a.lk - 1);
      rk[c] = ld16(kb_ + (long)key * a.k_ld + cc * CH);
    }
#pragma unroll
    for (int c = 0; c < V_CH; ++c) {
      const int id = c * NT + tid;
      const int r = id / (KVT / CH), cc = id % (KVT / CH);
      rv[c] = ld16(vb_ + (long)r * a.vt_ld + kv0 + cc * CH);
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int c = 0; c < K_CH; ++c) {
      const int id = c * NT + tid;
      const int r = id / (DH / CH), cc = id % (DH / CH);
      st16(&sK[buf][r * KLD + cc * CH], rk[c]);
    }
#pragma unroll
    for (int c = 0; c < V_CH; ++c) {
      const int id = c * NT + tid;
      const int r = id / (KVT / CH), cc = id % (KVT / CH);
      // groups of 4 consecutive keys stay contiguous under the permutation
      const T* src = reinterpret_cast<const T*>(&rv[c]);
#pragma unroll
      for (int g = 0; g < CH / 4; ++g) {
        const int key = cc * CH + 4 * g;            // key inside the tile
        const int w = key & 31;
        const int pos = (key & ~31) + 16 * ((w >> 2) & 1) + 4 * (w >> 3);
        T* dst = &sV[buf][r * VLD + pos];
        if (sizeof(T) == 2) {
          *reinterpret_cast<uint2*>(dst) = *reinterpret_cast<const uint2*>(src + 4 * g);
        } else {
          *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(src + 4 * g);
        }
      }
    }
  };

  f32x16 o[QB][NDT];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[qb][dt][r] = 0.0f;
  float m_run[QB], l_run[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) { m_run[qb] = -INFINITY; l_run[qb] = 0.0f; }

  const int ntiles = (a.lk + KVT - 1) / KVT;
  load_tile(0);
  store_tile(0);
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int cur = t & 1;
    const int kv0 = t * KVT;
    const bool more = t + 1 < ntiles;
    if (more) load_tile(kv0 + KVT);

    // S^T = K Q^T
    f32x16 sc[NKT][QB];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int r = 0; r < 16; ++r) sc[kt][qb][r] = 0.0f;
    const T* pk = &sK[cur][l32 * KLD + KPL * half];
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        typename MF::frag kf = MF::load(pk + kt * 32 * KLD + ks * KSTEP);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) sc[kt][qb] = MF::mma(kf, qf[qb][ks], sc[kt][qb]);
      }
    }
    if (kv0 + KVT > a.lk) {
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kv0 + kt * 32 + acc_row(r, lane);
          if (key >= a.lk)
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) sc[kt][qb][r] = -INFINITY;
        }
    }

    // online softmax; P^T packed into B-operand fragments.  The running
    // maximum is only raised (and O, l rescaled) when some lane's tile
    // maximum exceeds it by more than RESCALE_LOG2; otherwise the stale
    // maximum is kept and probabilities may reach 2^RESCALE_LOG2, which fp32
    // accumulation and the bf16 operand carry without loss of relative
    // precision.  The branch is uniform across the wave.
    typename MF::frag pf[QB][NKT][NPS];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[kt][qb][r]);
      mx = max_lane_pair32(mx) * a.scale_log2;
      if (__any(mx > m_run[qb] + RESCALE_LOG2)) {
        const float m_new = fmaxf(m_run[qb], mx);
        const float alpha = __builtin_amdgcn_exp2f(m_run[qb] - m_new);
        m_run[qb] = m_new;
        l_run[qb] *= alpha;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[qb][dt][r] *= alpha;
      }
      const float m_cur = m_run[qb];
      float lsum = 0.0f;
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        float p[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) p[r] = __builtin_amdgcn_exp2f(fmaf(sc[kt][qb][r], a.scale_log2, -m_cur));
#pragma unroll
        for (int ps = 0; ps < NPS; ++ps) {
          if constexpr (KPL == 1) {
            pf[qb][kt][ps] = to_t<T>(p[ps]);
            lsum += p[ps];
          } else {
            // the row sum is taken over the rounded operand that the value
            // product consumes, two elements per dot instruction
            typename MF::frag f;
#pragma unroll
            for (int i = 0; i < KPL; ++i) f[i] = to_t<T>(p[ps * KPL + i]);
            pf[qb][kt][ps] = f;
            const bf16x2 one = {(bf16)1.0f, (bf16)1.0f};
#pragma unroll
            for (int i = 0; i < KPL; i += 2) {
              const bf16x2 pr = {f[i], f[i + 1]};
              lsum = __builtin_amdgcn_fdot2_f32_bf16(pr, one, lsum, false);
            }
          }
        }
      }
      l_run[qb] += lsum;
    }

    // O^T += V^T P^T
    const T* pv = &sV[cur][l32 * VLD + 16 * half];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int ps = 0; ps < NPS; ++ps)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          typename MF::frag vf = MF::load(pv + dt * 32 * VLD + kt * 32 + ps * KPL);
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) o[qb][dt] = MF::mma(vf, pf[qb][kt][ps], o[qb][dt]);
        }

    if (more) store_tile(cur ^ 1);
    __syncthreads();
  }

  // normalise and store O[q][head*DH + channel]
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float l_tot = l_run[qb] + __shfl_xor(l_run[qb], 32, WAVE);
    const float inv = 1.0f / l_tot;
    const int row = q0 + qb * 32 + l32;
    if (row < a.lq) {
      T* dst = a.o + (long)s * a.o_ss + (long)row * a.o_ld + head * DH;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int ch = dt * 32 + 8 * g + 4 * half;
#pragma unroll
          for (int r = 0; r < 4; ++r) dst[ch + r] = to_t<T>(o[qb][dt][4 * g + r] * inv);
        }
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 variant with direct global->LDS tile loads.
//
// K and V^T tiles of KVT keys travel from global memory straight into a ring
// of STAGES LDS buffers by buffer loads (no staging registers, no LDS store
// instructions; keys past lk arrive as zeros);
// tile t+STAGES-1 is requested while tile t is processed, and one barrier per
// tile separates the reads of a buffer from its refill.  Rows are unpadded;
// 16-byte chunks are XOR-swizzled so that the fragment reads are free of bank
// conflicts.
//
// V^T is stored in natural key order.  The key order of P^T in the
// accumulators is made to match it instead: the score product reads, for its
// output row u, K row pi(u), where pi swaps bits 2 and 3 of u.  Accumulator
// register j of lane l holds output row u = 8(j/4) + 4(l/32) + j%4, so it
// holds key pi(u) = 16(j/8) + 8(l/32) + j%8, which is exactly element j%8 of
// k-step j/8 of the value product's B operand for lane l.  The K swizzle is
// taken in pi-space, f(r) = swz(pi(r)), so the permuted reads stay
// conflict-free.
// ---------------------------------------------------------------------------
CS_DEV int swap_bits23(int u) { return (u & ~12) | ((u & 4) << 1) | ((u & 8) >> 1); }

template <int DH, int QB, int KVT, int NW, int OCC, int STAGES, bool CROSS>
__global__ __launch_bounds__(64 * NW, OCC) void k_flash_dl(AttnArgs<bf16> a) {
  typedef Mfma32<bf16> MF;
  constexpr int KSTEP = MF::KSTEP;             // 16 keys / channels per MFMA step
  constexpr int CPR_K = DH / 8, RPI_K = 64 / CPR_K;    // K: chunks per row, rows per load
  constexpr int CPR_V = KVT / 8, RPI_V = 64 / CPR_V;   // V^T
  constexpr int K_INST = KVT / RPI_K / NW, V_INST = DH / RPI_V / NW;
  constexpr int PER_TILE = K_INST + V_INST;    // load instructions per wave per tile
  constexpr int K_ELEMS = KVT * DH, STAGE = 2 * KVT * DH;
  constexpr int NKT = KVT / 32, NDT = DH / 32, NKS = DH / KSTEP, NPS = 32 / KSTEP;
  static_assert(K_INST * RPI_K * NW == KVT && V_INST * RPI_V * NW == DH, "tile split");
  static_assert(STAGES >= 3 && STAGES <= 4, "ring depth");
  __shared__ __attribute__((aligned(1024))) bf16 smem[STAGES * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  constexpr int QPW = QB * 32;                 // queries per wave
  const int n_qt = (a.lq + NW * QPW - 1) / (NW * QPW);
  const int vid = xcd_contiguous(blockIdx.x, gridDim.x);
  const int qt = vid % n_qt, hs = vid / n_qt;
  const int head = hs % a.heads, s = hs / a.heads;
  const int kvs = a.kv_sel ? a.kv_sel[s] : s;
  const int q0 = qt * (NW * QPW) + wave * QPW;

  const bf16* qb_ = a.q + (long)s * a.q_ss + head * DH;
  const bf16* kb_ = a.k + (long)kvs * a.k_ss + head * DH;
  const bf16* vb_ = a.vt + (long)kvs * a.vt_ss + (long)head * DH * a.vt_ld;

  // Q^T fragments (B operand), kept for the whole key loop
  typename MF::frag qf[QB][NKS];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int row = min(q0 + qb * 32 + l32, a.lq - 1);
    const bf16* src = qb_ + (long)row * a.q_ld + MF::KPL * half;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      qf[qb][ks] = MF::load(src + ks * KSTEP);
      asm volatile("" : "+v"(qf[qb][ks]));
    }
  }

  // per-lane load sources: lane covers row (lane / CPR) of its instruction's
  // rows and physical chunk lane % CPR, i.e. logical chunk phys ^ f(row)
  // Buffer ranges: the lk key rows of this (stream, head), and its DH rows
  // of V^T (padded key length); keys past lk load as zeros and are masked.
  const int k_bytes = (int)(((long)(a.lk - 1) * a.k_ld + DH) * 2);
  const int v_bytes = (int)((long)DH * a.vt_ld * 2);
  int k_off[K_INST], v_off[V_INST];
#pragma unroll
  for (int i = 0; i < K_INST; ++i) {
    const int row = (wave * K_INST + i) * RPI_K + lane / CPR_K;
    k_off[i] = (row * (int)a.k_ld + ((lane % CPR_K) ^ chunk_swz<CPR_K>(swap_bits23(row))) * 8) * 2;
  }
#pragma unroll
  for (int i = 0; i < V_INST; ++i) {
    const int row = (wave * V_INST + i) * RPI_V + lane / CPR_V;
    v_off[i] = (row * (int)a.vt_ld + ((lane % CPR_V) ^ chunk_swz<CPR_V>(row)) * 8) * 2;
  }
  auto issue = [&](int tile, int st) {
    const int kv0 = tile * KVT;
    bf16* sk = smem + st * STAGE;
    bf16* sv = sk + K_ELEMS;
#pragma unroll
    for (int i = 0; i < K_INST; ++i)
      buffer_load_lds16(kb_, k_bytes, sk + (wave * K_INST + i) * RPI_K * DH, k_off[i],
                        kv0 * (int)a.k_ld * 2);
#pragma unroll
    for (int i = 0; i < V_INST; ++i)
      buffer_load_lds16(vb_, v_bytes, sv + (wave * V_INST + i) * RPI_V * KVT, v_off[i], kv0 * 2);
  };

  f32x16 o[QB][NDT];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[qb][dt][r] = 0.0f;
  float m_run[QB], l_run[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) { m_run[qb] = -INFINITY; l_run[qb] = 0.0f; }

  const int ntiles = (a.lk + KVT - 1) / KVT;
#pragma unroll
  for (int t = 0; t < STAGES - 1; ++t)
    if (t < ntiles) issue(t, t);

  // fragment rows: the score product reads K row pi(l32) of each 32-key
  // block; the value product reads V^T row (channel) l32 of each 32-block
  const int k_frag_row = swap_bits23(l32);

  for (int t = 0; t < ntiles; ++t) {
    // tile t has landed once at most min(rem, STAGES-2) later tiles are in flight
    const int rem = ntiles - 1 - t;
    if (rem >= STAGES - 2) wait_vm_barrier<(STAGES - 2) * PER_TILE>();
    else if (STAGES == 4 && rem == 1) wait_vm_barrier<PER_TILE>();
    else wait_vm_barrier<0>();
    if (t + STAGES - 1 < ntiles) issue(t + STAGES - 1, (t + STAGES - 1) % STAGES);
    const bf16* sk = smem + (t % STAGES) * STAGE;
    const bf16* sv = sk + K_ELEMS;
    const int kv0 = t * KVT;

    // S^T = K Q^T (rows in pi order)
    f32x16 sc[NKT][QB];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int r = 0; r < 16; ++r) sc[kt][qb][r] = 0.0f;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        const int row = kt * 32 + k_frag_row;
        const int c = 2 * ks + half;
        typename MF::frag kf = MF::load(sk + row * DH + (c ^ chunk_swz<CPR_K>(kt * 32 + l32)) * 8);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) sc[kt][qb] = MF::mma(kf, qf[qb][ks], sc[kt][qb]);
      }
    }
    // every V^T fragment of the tile is requested before the softmax, whose
    // arithmetic then hides the read latency of the value product
    typename MF::frag vf[NKT][NPS][NDT];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int ps = 0; ps < NPS; ++ps)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          const int row = dt * 32 + l32;
          const int c = 4 * kt + 2 * ps + half;
          vf[kt][ps][dt] = MF::load(sv + row * KVT + (c ^ chunk_swz<CPR_V>(row)) * 8);
        }
    if (kv0 + KVT > a.lk) {
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kv0 + kt * 32 + swap_bits23(acc_row(r, lane));
          if (key >= a.lk)
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) sc[kt][qb][r] = -INFINITY;
        }
    }

    // online softmax with lazy rescaling (see k_flash); P^T packed into
    // B-operand fragments, row sums over the rounded operands
    typename MF::frag pf[QB][NKT][NPS];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[kt][qb][r]);
      mx = max_lane_pair32(mx) * a.scale_log2;
      if (__any(mx > m_run[qb] + RESCALE_LOG2)) {
        const float m_new = fmaxf(m_run[qb], mx);
        const float alpha = __builtin_amdgcn_exp2f(m_run[qb] - m_new);
        m_run[qb] = m_new;
        l_run[qb] *= alpha;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[qb][dt][r] *= alpha;
      }
      float lsum = 0.0f;
      const bf16x2 one = {(bf16)1.0f, (bf16)1.0f};
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        float p[16];
#pragma unroll
        for (int r = 0; r < 16; ++r)
          p[r] = __builtin_amdgcn_exp2f(fmaf(sc[kt][qb][r], a.scale_log2, -m_run[qb]));
#pragma unroll
        for (int ps = 0; ps < NPS; ++ps) {
          typename MF::frag f;
#pragma unroll
          for (int i = 0; i < 8; ++i) f[i] = (bf16)p[ps * 8 + i];
          pf[qb][kt][ps] = f;
#pragma unroll
          for (int i = 0; i < 8; i += 2) {
            const bf16x2 pr = {f[i], f[i + 1]};
            lsum = __builtin_amdgcn_fdot2_f32_bf16(pr, one, lsum, false);
          }
        }
      }
      l_run[qb] += lsum;
    }

    // O^T += V^T P^T
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int ps = 0; ps < NPS; ++ps)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) o[qb][dt] = MF::mma(vf[kt][ps][dt], pf[qb][kt][ps], o[qb][dt]);
  }

  // normalise and store O[q][head*DH + channel]
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float l_tot = l_run[qb] + __shfl_xor(l_run[qb], 32, WAVE);
    const float inv = 1.0f / l_tot;
    const int row = q0 + qb * 32 + l32;
    if (row < a.lq) {
      bf16* dst = a.o + (long)s * a.o_ss + (long)row * a.o_ld + head * DH;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int ch = dt * 32 + 8 * g + 4 * half;
          bf16x4 q;
#pragma unroll
          for (int r = 0; r < 4; ++r) q[r] = (bf16)(o[qb][dt][4 * g + r] * inv);
          *reinterpret_cast<bf16x4*>(dst + ch) = q;
        }
    }
  }
}


// ---------------------------------------------------------------------------
// bf16 variant with padded LDS rows (head dims 64 and 128).
//
// The direct loads place any 16-byte chunk of global memory anywhere in the
// 1 KB an instruction fills, so the tiles are stored with padded rows instead
// of a swizzle: a K row of DH/8 chunks takes DH/8 + 1 chunk slots and a V^T
// row of 8 chunks takes 9.  The extra slot of a row receives a copy of the
// row's last chunk (same cache line, no extra traffic) and is never read.
// Row strides of 272 and 144 bytes spread 16 consecutive rows over all 64
// banks, and since no chunk index is permuted every fragment read of a tile is
// one base register plus a compile-time offset: the per-read address
// arithmetic of the swizzled layout disappears from the key loop.  Stage t of
// the ring holds K (64 x 17 chunks = 17 KB) then V^T (DH x 9 chunks), all
// whole 1 KB load instructions, spread over the waves (the first few waves
// issue one more than the others).  Results are bitwise those of k_flash_dl.
//
// Occupancy.  The V^T fragments are read inside the value product, each just
// before its two MFMAs, instead of all ahead of the softmax: that saves 64
// registers and brings a wave to 160, so three waves fit per SIMD (12 waves
// of 32 queries per workgroup).  The third wave hides LDS latency better than
// the early reads did (measured 4% faster at 32,760 tokens).
// ---------------------------------------------------------------------------
template <int DH, int NW, int OCC, int STAGES, bool CROSS>
__global__ __launch_bounds__(64 * NW, OCC) void k_flash_pad(AttnArgs<bf16> a) {
  typedef Mfma32<bf16> MF;
  typedef typename MF::frag frag;
  constexpr int KVT = 64, KSTEP = MF::KSTEP;
  constexpr int CK = DH / 8 + 1, CV = KVT / 8 + 1;   // chunk slots per padded row
  constexpr int KRS = CK * 16, VRS = CV * 16;        // padded row strides (bytes)
  constexpr int K_INSTR = KVT * CK / 64, V_INSTR = DH * CV / 64;
  static_assert(K_INSTR * 64 == KVT * CK && V_INSTR * 64 == DH * CV, "whole 1 KB loads");
  constexpr int KB = K_INSTR * 1024, STAGE = KB + V_INSTR * 1024;
  constexpr int TOT = K_INSTR + V_INSTR;             // load instructions per tile
  constexpr int NPW = (TOT + NW - 1) / NW;           // per wave, for the first NBUSY waves
  constexpr int NBUSY = TOT - (NPW - 1) * NW;        // the others issue NPW - 1
  constexpr int NKT = KVT / 32, NDT = DH / 32, NKS = DH / KSTEP, NPS = 32 / KSTEP;
  static_assert(STAGES >= 3 && STAGES <= 4, "ring depth");
  __shared__ __attribute__((aligned(1024))) char smem[STAGES * STAGE];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: loads use SGPR ranges
  const int half = lane >> 5, l32 = lane & 31;
  const int n_qt = (a.lq + NW * 32 - 1) / (NW * 32);
  const int vid = xcd_contiguous(blockIdx.x, gridDim.x);
  const int qt = vid % n_qt, hs = vid / n_qt;
  const int head = hs % a.heads, s = hs / a.heads;
  const int kvs = a.kv_sel ? a.kv_sel[s] : s;
  const int q0 = qt * (NW * 32) + wave * 32;

  const bf16* qb_ = a.q + (long)s * a.q_ss + head * DH;
  const bf16* kb_ = a.k + (long)kvs * a.k_ss + head * DH;
  const bf16* vb_ = a.vt + (long)kvs * a.vt_ss + (long)head * DH * a.vt_ld;

  // Q^T fragments (B operand), kept for the whole key loop
  frag qf[NKS];
  {
    const int row = min(q0 + l32, a.lq - 1);
    const bf16* src = qb_ + (long)row * a.q_ld + MF::KPL * half;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      qf[ks] = MF::load(src + ks * KSTEP);
      asm volatile("" : "+v"(qf[ks]));
    }
  }

  // load instruction i of this wave fills slots [64g, 64g + 64) of the stage,
  // g = wave + NW*i; slot p of the K part is row p / CK, chunk p % CK (the
  // padding slot takes the row's last chunk), likewise for V^T.  Keys past
  // lk load as zeros (K range) or are finite padding (V^T) and are masked.
  const int k_bytes = (int)(((long)(a.lk - 1) * a.k_ld + DH) * 2);
  const int v_bytes = (int)((long)DH * a.vt_ld * 2);
  int voff[NPW];
#pragma unroll
  for (int i = 0; i < NPW; ++i) {
    const int g = wave + NW * i;
    if (g < K_INSTR) {
      const int p = g * 64 + lane, row = p / CK, ch = min(p % CK, CK - 2);
      voff[i] = (row * (int)a.k_ld + ch * 8) * 2;
    } else {
      const int p = (g - K_INSTR) * 64 + lane, row = p / CV, ch = min(p % CV, CV - 2);
      voff[i] = (row * (int)a.vt_ld + ch * 8) * 2;
    }
  }
  const bool busy = wave < NBUSY;
  auto issue = [&](int tile, int st) {
    const int kv0 = tile * KVT;
    char* base = smem + st * STAGE;
#pragma unroll
    for (int i = 0; i < NPW; ++i) {
      const int g = wave + NW * i;
      if (i < NPW - 1 || busy) {
        if (g < K_INSTR)
          buffer_load_lds16(kb_, k_bytes, base + g * 1024, voff[i], kv0 * (int)a.k_ld * 2);
        else
          buffer_load_lds16(vb_, v_bytes, base + g * 1024, voff[i], kv0 * 2);
      }
    }
  };

  f32x16 o[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[dt][r] = 0.0f;
  float m_run = -INFINITY, l_run = 0.0f;

  const int ntiles = (a.lk + KVT - 1) / KVT;
#pragma unroll
  for (int t = 0; t < STAGES - 1; ++t)
    if (t < ntiles) issue(t, t);

  // fragment bases: the score product reads K row pi(l32) of each 32-key
  // block (pi swaps bits 2 and 3, see k_flash_dl), the value product V^T row
  // (channel) l32 of each 32-channel block
  const int lane_k = swap_bits23(l32) * KRS + half * 16;
  const int lane_v = KB + l32 * VRS + half * 16;
  const bf16x2 one = {(bf16)1.0f, (bf16)1.0f};

  for (int t = 0; t < ntiles; ++t) {
    // tile t has landed once at most min(rem, STAGES-2) later tiles are in flight
    const int inflight = min(ntiles - 1 - t, STAGES - 2);
    if (busy) {
      if (inflight >= 2) wait_vm_barrier<2 * NPW>();
      else if (inflight == 1) wait_vm_barrier<NPW>();
      else wait_vm_barrier<0>();
    } else {
      if (inflight >= 2) wait_vm_barrier<2 * (NPW - 1)>();
      else if (inflight == 1) wait_vm_barrier<NPW - 1>();
      else wait_vm_barrier<0>();
    }
    if (t + STAGES - 1 < ntiles) issue(t + STAGES - 1, (t + STAGES - 1) % STAGES);
    const char* pk = smem + (t % STAGES) * STAGE + lane_k;
    const char* pv = smem + (t % STAGES) * STAGE + lane_v;
    const int kv0 = t * KVT;

    // S^T = K Q^T (rows in pi order)
    f32x16 sc[NKT];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) sc[kt][r] = 0.0f;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        frag kf = MF::load(reinterpret_cast<const bf16*>(pk + kt * 32 * KRS + ks * 32));
        sc[kt] = MF::mma(kf, qf[ks], sc[kt]);
      }
    if (kv0 + KVT > a.lk) {
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kv0 + kt * 32 + swap_bits23(acc_row(r, lane));
          if (key >= a.lk) sc[kt][r] = -INFINITY;
        }
    }

    // online softmax with lazy rescaling (see k_flash)
    frag pf[NKT][NPS];
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[kt][r]);
    mx = max_lane_pair32(mx) * a.scale_log2;
    if (__any(mx > m_run + RESCALE_LOG2)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;
    }
    float lsum = 0.0f;
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt) {
      float p[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) p[r] = __builtin_amdgcn_exp2f(fmaf(sc[kt][r], a.scale_log2, -m_run));
#pragma unroll
      for (int ps = 0; ps < NPS; ++ps) {
        frag f;
#pragma unroll
        for (int i = 0; i < 8; ++i) f[i] = (bf16)p[ps * 8 + i];
        pf[kt][ps] = f;
#pragma unroll
        for (int i = 0; i < 8; i += 2) {
          const bf16x2 pr = {f[i], f[i + 1]};
          lsum = __builtin_amdgcn_fdot2_f32_bf16(pr, one, lsum, false);
        }
      }
    }
    l_run += lsum;

    // O^T += V^T P^T, each V^T fragment read just before its product
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int ps = 0; ps < NPS; ++ps)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          const frag vf = MF::load(reinterpret_cast<const bf16*>(pv + dt * 32 * VRS + kt * 64 + ps * 32));
          o[dt] = MF::mma(vf, pf[kt][ps], o[dt]);
        }
  }

  // normalise and store O[q][head*DH + channel]
  const float l_tot = l_run + __shfl_xor(l_run, 32, WAVE);
  const float inv = 1.0f / l_tot;
  const int row = q0 + l32;
  if (row < a.lq) {
    bf16* dst = a.o + (long)s * a.o_ss + (long)row * a.o_ld + head * DH;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int ch = dt * 32 + 8 * g + 4 * half;
        bf16x4 q;
#pragma unroll
        for (int r = 0; r < 4; ++r) q[r] = (bf16)(o[dt][4 * g + r] * inv);
        *reinterpret_cast<bf16x4*>(dst + ch) = q;
      }
  }
}

}  // namespace cs
