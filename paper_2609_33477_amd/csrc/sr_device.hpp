// Device-side helpers shared by the replay kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sr_internal.hpp"

namespace sr {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Storage tags: bf16 and fp8 tensors are handled as raw bits.
struct bf16_t { uint16_t bits; };
struct fp8_t { uint8_t bits; };

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) {
  return __uint_as_float(h << 16);
}

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two fp32 -> packed bf16 (a in the low half), round to nearest even: one
// v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  return (uint16_t)(pack_bf16x2(f, 0.f) & 0xffffu);
}

// OCP FP8 E4M3 -> bf16 bits, exact.  Normal: 2^(e-7) (1 + m/8); subnormal:
// m 2^-9; e = 15, m = 7 is NaN.
__device__ __forceinline__ uint32_t e4m3_to_bf16_bits(uint32_t b) {
  const uint32_t s = (b & 0x80u) << 8;
  const uint32_t e = (b >> 3) & 0xfu;
  const uint32_t m = b & 0x7u;
  if (e == 0) {
    if (m == 0) return s;
    // m * 2^-9 with m in 1..7: normalise the leading bit.
    const uint32_t lead = 31u - __builtin_clz(m);           // 0..2
    const uint32_t exp = 127u - 9u + lead;                    // biased bf16 exponent
    const uint32_t mant = (m << (7u - lead)) & 0x7fu;
    return s | (exp << 7) | mant;
  }
  if (e == 15 && m == 7) return s | 0x7fc0u;
  return s | ((e + 120u) << 7) | (m << 4);
}

__device__ __forceinline__ float e4m3_to_f32(uint32_t b) {
  return bf16_bits_to_f32(e4m3_to_bf16_bits(b));
}

// Generic scalar load/store of a storage element as fp32.
template <typename T> struct Elem;
template <> struct Elem<float> {
  static constexpr int bytes = 4;
  __device__ static float load(const void* p, int64_t i) { return static_cast<const float*>(p)[i]; }
  __device__ static void store(void* p, int64_t i, float v) { static_cast<float*>(p)[i] = v; }
};
template <> struct Elem<bf16_t> {
  static constexpr int bytes = 2;
  __device__ static float load(const void* p, int64_t i) {
    return bf16_bits_to_f32(static_cast<const uint16_t*>(p)[i]);
  }
  __device__ static void store(void* p, int64_t i, float v) {
    static_cast<uint16_t*>(p)[i] = f32_to_bf16_bits(v);
  }
};
template <> struct Elem<fp8_t> {
  static constexpr int bytes = 1;
  __device__ static float load(const void* p, int64_t i) {
    return e4m3_to_f32(static_cast<const uint8_t*>(p)[i]);
  }
};

// ---------------------------------------------------------------------------
// MFMA 32x32 tiles.  Accumulator layout (both variants): lane l, register r
// holds C[8*(r/4) + 4*(l/32) + (r%4)][l%32].  Operand layout: lane l supplies
// A[l%32][k-slots] and B[k-slots][l%32]; the 32x32x16 bf16 form takes 8
// consecutive k per lane (lanes 0-31: k 0-7, lanes 32-63: k 8-15), the
// 32x32x2 f32 form one k per lane (lanes 0-31: k 0, lanes 32-63: k 1).
// ---------------------------------------------------------------------------
template <typename OP> struct Mfma;

template <> struct Mfma<bf16_t> {
  static constexpr int K = 16;      // k per instruction
  static constexpr int HALF = 8;    // k per lane
  typedef bf16x8 frag;
  __device__ static void mma(f32x16& c, const frag& a, const frag& b) {
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};

template <> struct Mfma<float> {
  static constexpr int K = 2;
  static constexpr int HALF = 1;
  typedef float frag;
  __device__ static void mma(f32x16& c, const frag& a, const frag& b) {
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

// Workgroup barrier that waits only for this wave's LDS traffic (lgkmcnt),
// not for outstanding global loads, so register prefetches stay in flight
// across it.  s_waitcnt immediate: vmcnt and expcnt at their maxima, lgkmcnt 0.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xc07f);
  __builtin_amdgcn_s_barrier();
}

// 16 bytes per lane, global -> LDS at lds_base + 16 * lane (wave-uniform
// base).  Inline asm: the compiler would otherwise wait for every such load
// before any later LDS read; completion is tracked by hand (wait_vm) before
// the barrier that publishes a stage.
// `lds_off` must be wave-uniform (it is an SGPR operand).
__device__ __forceinline__ void dma16(const void* src, uint32_t lds_off) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds_off), "v"(src) : "memory", "m0");
}

// The same with a wave-uniform 64-bit base in SGPRs and a 32-bit per-lane
// byte offset (the instruction's saddr form): no 64-bit address arithmetic
// per lane.
__device__ __forceinline__ void dma16_s(const void* sbase, uint32_t voff, uint32_t lds_off) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds_off), "v"(voff), "s"(sbase)
               : "memory", "m0");
}

// s_waitcnt vmcnt(N) with lgkmcnt and expcnt left at their maxima
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__device__ __forceinline__ int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

// ds_read_b64_tr_b16: lane i of each 16-lane group receives rows
// kbase .. kbase + 3 of column n0 + i (4 bf16) when lane j of the group
// addresses row kbase + j / 4, columns n0 + 4 (j % 4) .. + 3.
__device__ __forceinline__ uint2 lds_tr4(const __attribute__((address_space(3))) char* p) {
  typedef short v4s __attribute__((ext_vector_type(4)));
  const v4s v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s*)p);
  return __builtin_bit_cast(uint2, v);
}

// Work units are ordered longest segment first, so the longest serial chain
// starts first.  Returns the segment holding `rank` when the live segments
// are ordered by descending length (ties by index, sentinel segments last);
// the natural order above kSortMax segments.  Every thread of the block must
// call it: it ends with a barrier.  A: any argument block with n_seg, cu and
// slot_ids.
constexpr int kSortMax = 256;
template <typename A>
__device__ int segment_of_rank(const A& a, int rank, int* shared_sel) {
  if (a.n_seg > kSortMax) return rank;
  auto len = [&](int s) -> int {
    const int slot = a.slot_ids ? a.slot_ids[s] : s;
    return slot < 0 ? -1 : a.cu[s + 1] - a.cu[s];
  };
  for (int s = threadIdx.x; s < a.n_seg; s += blockDim.x) {
    const int ls = len(s);
    int r = 0;
    for (int s2 = 0; s2 < a.n_seg; ++s2) {
      const int l2 = len(s2);
      r += (l2 > ls) || (l2 == ls && s2 < s);
    }
    if (r == rank) *shared_sel = s;
  }
  __syncthreads();
  return *shared_sel;
}

}  // namespace sr
