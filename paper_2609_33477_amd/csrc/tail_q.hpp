// Conv tail, q part, for bf16 anchors (Appendix A: the conv state is the last
// w-1 inputs of the q, k, v channels).  W_q is used nowhere else in
// state-only replay, so the q projections of each segment's last w-1 rows are
// one small GEMM over the gathered tail rows of all segments x the q
// channels.  These blocks ride in the fused projection's grid after its
// tiles: they are dispatched into its last, partial round (or onto CUs its
// tiles leave idle), so the tail costs no launch of its own.
//
// Block (8 waves): 32 tail rows x 32 q channels, on v_mfma_f32_32x32x16_bf16.
// Anchor rows and W_q rows go global -> LDS by DMA in contiguous 1 KB runs
// per row (a whole row of the 512-column stage per instruction), two stages
// in flight, 16-byte chunks XOR-swizzled by (row & 15) so the fragment reads
// are conflict free; each wave takes a share of every stage's k-steps and the
// waves add their accumulators through LDS.  Staging whole rows keeps the
// load path at its per-CU rate: fragment-shaped global loads (32 rows x 32
// bytes per instruction) ran at about a quarter of it.  The block writes the
// q projection of each live tail row and zeros at positions before a
// segment's first row.  One more block per 32 tail rows writes those leading
// zeros for the channels past the q ones, whose rows the projection's
// epilogue writes.
#pragma once

#include <type_traits>

#include "sr_device.hpp"

namespace sr {

constexpr int kTqWaves = 8;
constexpr int kTqChunk = 512;                  // d_model columns per stage
constexpr int kTqHalf = 32 * 1024;             // 32 rows x 1 KB
constexpr int kTqStage = 2 * kTqHalf;          // anchor rows | weight rows
constexpr int kTqTables = 2 * kTqStage;        // row tables after the two stages
constexpr int kTqLds = kTqTables + 32 * 16;    // bytes of LDS a block uses

// Tail row r = (segment r / (w-1), position r % (w-1)) -> anchor row, or -1
// when the position precedes the segment's first row or the slot is a
// sentinel.
__device__ __forceinline__ int64_t tail_row(const TailArgs& a, int r, int* slot, int* pos) {
  const int w1 = a.w - 1;
  const int b = r / w1;
  *pos = r - b * w1;
  *slot = a.slot_ids ? a.slot_ids[b] : b;
  const int64_t s0 = a.cu[b], s1 = a.cu[b + 1];
  const int64_t t = s1 - w1 + *pos;
  return (*slot >= 0 && t >= s0) ? t : -1;
}

__device__ __forceinline__ int tq_swz(int m) { return m & 15; }

__device__ __forceinline__ void tq_store(const TailArgs& a, int64_t i, float v) {
  if (a.tail_bf16) static_cast<uint16_t*>(a.tail)[i] = f32_to_bf16_bits(v);
  else static_cast<float*>(a.tail)[i] = v;
}

// Block (bx, by) of the q-tail grid (tail_q_grid_x/y); smem holds kTqLds
// bytes.  Every thread of a 64 * kTqWaves-thread block calls it.  TW: W_q
// storage (bf16_t, or fp8_t converted exactly to bf16 after the LDS read,
// scaled per channel by s_q at the end).
template <typename TW>
__device__ __forceinline__ void tail_q_block(const TailArgs& a, int bx, int by, char* smem) {
  typedef __attribute__((address_space(3))) char lchar;
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
  int* row_slot = reinterpret_cast<int*>(smem + kTqTables);   // per tail row of the block: slot (< 0: none)
  int* row_pos = row_slot + 32;                                // position (< 0: -1 - position, zero)
  int64_t* row_t = reinterpret_cast<int64_t*>(row_pos + 32);   // anchor row (0 for dead rows)
  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int R = a.n_seg * (a.w - 1), w1 = a.w - 1;
  const int nqb = (a.c_q + 31) / 32;
  if (threadIdx.x < 32) {
    const int rr = by * 32 + threadIdx.x;
    int sl = -1, ps = 0;
    int64_t t = -1;
    if (rr < R) t = tail_row(a, rr, &sl, &ps);
    row_slot[threadIdx.x] = sl;
    row_pos[threadIdx.x] = t >= 0 ? ps : -1 - ps;
    row_t[threadIdx.x] = t >= 0 ? t : 0;
  }
  __syncthreads();
  if (bx == nqb) {
    // channels [c_q, c_tail): zeros at positions before each segment's first row
    const int nc = a.c_tail - a.c_q;
    for (int i = 0; i < 32; ++i) {
      const int sl = row_slot[i], pp = row_pos[i];
      if (sl < 0 || pp >= 0) continue;
      for (int col = threadIdx.x; col < nc; col += 64 * kTqWaves)
        tq_store(a, ((int64_t)sl * a.c_tail + a.c_q + col) * w1 + (-1 - pp), 0.f);
    }
    return;
  }
  constexpr int EB = sizeof(TW);            // weight bytes per element
  constexpr int WDMA = 2 * EB;              // weight DMAs per wave per stage: 4 (bf16, one row each), 2 (fp8, two rows)
  constexpr int DPW = 4 + WDMA;             // DMAs per wave per stage
  const int c0 = bx * 32;
  const int D = a.D;
  const uint32_t lds0 = (uint32_t)(uintptr_t)smem;
  const char* xbase = static_cast<const char*>(a.anchors);
  const char* wbase = static_cast<const char*>(a.w_q);
  // Stage ch: columns [512 ch, 512 ch + kc).  Row m's 16-byte chunk g sits at
  // LDS chunk g ^ swz(m); a lane whose LDS chunk lies past the stage's
  // columns loads the row's last chunk instead (never read).
  auto issue = [&](int ch) {
    const int k0 = ch * kTqChunk;
    const int kc = min(kTqChunk, D - k0);
    const uint32_t st = lds0 + (ch & 1) * kTqStage;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = 4 * wid + j;
      const int g = min(lane ^ tq_swz(m), kc / 8 - 1);
      dma16(xbase + (row_t[m] * D + k0) * 2 + g * 16, st + m * 1024);
    }
#pragma unroll
    for (int j = 0; j < WDMA; ++j) {
      int m, p;
      if constexpr (EB == 2) {
        m = 4 * wid + j;
        p = lane;
      } else {                                  // 512-byte fp8 rows: two per instruction
        m = 4 * wid + 2 * j + (lane >> 5);
        p = lane & 31;
      }
      const int c = min(c0 + m, a.c_q - 1);
      const int g = min(p ^ tq_swz(m), kc * EB / 16 - 1);
      dma16(wbase + ((int64_t)c * D + k0) * EB + g * 16,
            st + kTqHalf + (EB == 2 ? m * 1024 : (4 * wid + 2 * j) * 512));
    }
  };
  const int nch = (D + kTqChunk - 1) / kTqChunk;
  issue(0);
  if (nch > 1) issue(1);
  const int mm = lane & 31, h = lane >> 5;
  f32x16 acc = zero16();
  for (int ch = 0; ch < nch; ++ch) {
    // this wave's DMAs of stage ch have landed (those of ch + 1 may not);
    // after the barrier every wave's have
    if (ch + 1 < nch) wait_vm<DPW>();
    else wait_vm<0>();
    __builtin_amdgcn_s_barrier();
    const int ns = min(kTqChunk, D - ch * kTqChunk) / 16;
    const int s_lo = wid * ns / kTqWaves, s_hi = (wid + 1) * ns / kTqWaves;
    const lchar* st = (const lchar*)smem + (ch & 1) * kTqStage;
    for (int s = s_lo; s < s_hi; ++s) {
      const int chunk = 16 * ((2 * s + h) ^ tq_swz(mm));
      const bf16x8 av =
          as_bf16x8(__builtin_bit_cast(uint4, *reinterpret_cast<const __attribute__((address_space(3))) u32x4*>(
                                                  st + mm * 1024 + chunk)));
      bf16x8 wv;
      if constexpr (EB == 2) {
        wv = as_bf16x8(__builtin_bit_cast(
            uint4, *reinterpret_cast<const __attribute__((address_space(3))) u32x4*>(st + kTqHalf + mm * 1024 + chunk)));
      } else {
        const uint2 v = __builtin_bit_cast(uint2, *reinterpret_cast<const __attribute__((address_space(3))) u32x2*>(
                                                      st + kTqHalf + mm * 512 + 16 * (s ^ tq_swz(mm)) + 8 * h));
        uint4 o;
        o.x = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(v.x, 1.0f, false));
        o.y = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(v.x, 1.0f, true));
        o.z = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(v.y, 1.0f, false));
        o.w = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(v.y, 1.0f, true));
        wv = as_bf16x8(o);
      }
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, wv, acc, 0, 0, 0);
    }
    lds_barrier();   // every wave is done with this stage
    if (ch + 2 < nch) issue(ch + 2);
  }
  // the waves' partial sums meet in the drained stages
  float* part = reinterpret_cast<float*>(smem);   // [kTqWaves - 1][16][64]
  if (wid > 0) {
#pragma unroll
    for (int i = 0; i < 16; ++i) part[((wid - 1) * 16 + i) * 64 + lane] = acc[i];
  }
  __syncthreads();
  if (wid > 0) return;
#pragma unroll
  for (int w = 0; w < kTqWaves - 1; ++w)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[i] += part[(w * 16 + i) * 64 + lane];
  const int col = c0 + mm;
  if (col >= a.c_q) return;
  const float scale = std::is_same<TW, fp8_t>::value ? Elem<bf16_t>::load(a.s_q, col) : 1.f;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int ri = acc_row(i, lane);
    const int sl = row_slot[ri], pp = row_pos[ri];
    if (sl >= 0) tq_store(a, ((int64_t)sl * a.c_tail + col) * w1 + (pp >= 0 ? pp : -1 - pp), pp >= 0 ? acc[i] * scale : 0.f);
  }
}

}  // namespace sr
