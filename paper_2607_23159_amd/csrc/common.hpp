// Shared definitions for the gfx950 kernels and the runtime.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

typedef __bf16 bf16;
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

#define CS_DEV __device__ __forceinline__

constexpr int WAVE = 64;

// ---------------------------------------------------------------------------
// 32x32 MFMA family, per element type.
//   A operand (32 x KSTEP): lane l holds row l%32, k = KPL*(l/32) + i.
//   B operand (KSTEP x 32): lane l holds column l%32, k = KPL*(l/32) + i.
//   Accumulator (32 x 32, 16 floats): register j of lane l is
//     row 8*(j/4) + 4*(l/32) + (j%4), column l%32.
// bf16: v_mfma_f32_32x32x16_bf16 (8 values per lane, K = 16).
// fp32: v_mfma_f32_32x32x2_f32   (1 value per lane,  K = 2).
// ---------------------------------------------------------------------------
template <typename T> struct Mfma32;

template <> struct Mfma32<bf16> {
  static constexpr int KPL = 8;
  static constexpr int KSTEP = 16;
  typedef bf16x8 frag;
  static CS_DEV f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  static CS_DEV frag load(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }
};

template <> struct Mfma32<float> {
  static constexpr int KPL = 1;
  static constexpr int KSTEP = 2;
  typedef float frag;
  static CS_DEV f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  static CS_DEV frag load(const float* p) { return *p; }
};

// Accumulator register j -> row offset inside the 32x32 tile for lane l.
CS_DEV int acc_row(int j, int lane) { return 8 * (j >> 2) + 4 * (lane >> 5) + (j & 3); }

template <typename T> CS_DEV T to_t(float v);
template <> CS_DEV bf16 to_t<bf16>(float v) { return (bf16)v; }
template <> CS_DEV float to_t<float>(float v) { return v; }
template <typename T> CS_DEV float to_f(T v) { return (float)v; }

// 16-byte copy helpers.
struct alignas(16) Chunk16 { uint32_t w[4]; };
CS_DEV Chunk16 ld16(const void* p) { return *reinterpret_cast<const Chunk16*>(p); }
CS_DEV void st16(void* p, Chunk16 c) { *reinterpret_cast<Chunk16*>(p) = c; }

// GELU, tanh form: 0.5 x (1 + tanh(u)), u = sqrt(2/pi) (x + 0.044715 x^3).
// Since 0.5 (1 + tanh(u)) = 1 / (1 + e^(-2u)), it is evaluated as
// x / (1 + 2^(x (c1 + c3 x^2))) with c1 = -2 sqrt(2/pi) log2(e) and
// c3 = 0.044715 c1: two multiplies and a multiply-add for the exponent, the
// hardware exp2 and reciprocal, an add and a multiply (the tanh form took
// twice the VALU work).  Large |x| saturate correctly: 2^(+big) = inf gives
// x / inf = 0 for x < 0, 2^(-big) = 0 gives x for x > 0.
CS_DEV float gelu_tanh(float x) {
  const float c1 = -2.302208198144325f;           // -2 sqrt(2/pi) / ln(2)
  const float c3 = -0.1029432395800235f;          // 0.044715 * c1
  const float z = x * fmaf(x * x, c3, c1);        // -2 u log2(e)
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(z));
}
CS_DEV float silu(float x) { return x / (1.0f + expf(-x)); }

CS_DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
  return v;
}
CS_DEV double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
  return v;
}

// Maximum of x over lanes l and l ^ 32.  v_permlane32_swap exchanges the two
// 32-lane halves inside the VALU (no LDS round trip, unlike a shuffle).
CS_DEV float max_lane_pair32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// The dispatcher deals workgroups round-robin to the 8 XCDs, each with its
// own L2.  This maps a hardware workgroup id to a virtual id so that every
// XCD runs one contiguous range of virtual ids (a bijection on [0, nwg) for
// any nwg); consecutive virtual ids then share their operands in one L2.
CS_DEV int xcd_contiguous(int bid, int nwg) {
  const int per = nwg >> 3, rem = nwg & 7, x = bid & 7;
  return x * per + min(x, rem) + (bid >> 3);
}

// ---- direct global->LDS loads (gfx950 global_load_lds_dwordx4): each
// wave instruction moves 64 x 16 bytes into 1 KB of LDS at base + 16*lane,
// with an arbitrary global address per lane.
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void gbl_void_t;

// The same through the buffer path (buffer_load_dwordx4 ... lds): a raw
// buffer descriptor over [base, base + bytes) and a 32-bit per-lane byte
// offset voff plus a wave-uniform byte offset soff.  Lanes whose 16 bytes do
// not lie inside the range receive zeros without any memory access.  The
// address unit handles a 32-bit offset per lane instead of a 64-bit address,
// which measured 3-10% faster in the GEMM main loop.  Kept out of lambdas:
// the builtins exist for the device pass only.
__device__ __forceinline__ void buffer_load_lds16(const void* base, int bytes, void* lds, int voff,
                                                  int soff) {
  // dword 3 of the descriptor: 32-bit data format, no swizzle, raw access
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes,
                                                                     0x00020000);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t*)lds, 16, voff, soff, 0, 0);
}

// XOR swizzle of the 16-byte chunks of LDS rows that hold CPR chunks each:
// chunk c of row r is stored at c ^ chunk_swz(r), so that 16-byte reads of
// one logical chunk from 16 (or 8) consecutive rows hit distinct banks.
template <int CPR> CS_DEV int chunk_swz(int r) {
  static_assert(CPR == 2 || CPR == 4 || CPR == 8 || CPR == 16, "chunks per row");
  constexpr int LOG = CPR == 2 ? 1 : (CPR == 4 ? 2 : (CPR == 8 ? 3 : 4));
  return (r ^ (r >> LOG)) & (CPR - 1);
}

// Wait until at most n vector-memory operations of this wave are
// outstanding, then barrier; the memory clobber keeps the compiler from moving
// LDS accesses across it.
template <int n> CS_DEV void wait_vm_barrier() {
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(n) : "memory");
}

inline int cdiv(long a, long b) { return (int)((a + b - 1) / b); }
inline long round_up(long a, long b) { return (a + b - 1) / b * b; }
