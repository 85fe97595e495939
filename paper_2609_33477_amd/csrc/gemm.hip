// Plain bf16 GEMMs of a replayed transformer block (group replay chaining,
// Section 4.1), C = A B^T with A [M][K] row-major activations, B [N][K]
// row-major weights (nn.Linear layout), fp32 accumulation, and the block's
// element-wise work fused into the epilogue:
//   RESID   C[m][n] += acc          (fp32 residual stream, in place): the
//                                    output projection and the MLP's down
//                                    projection add into the hidden state
//   SWIGLU  H[m][j] = SiLU(gate) * up (bf16), gate = A W_gate^T,
//           up = A W_up^T: the tile's 32-column blocks alternate gate and up
//           rows of the same hidden units, so a lane holds both factors of
//           each output in matching registers.
//
// Main loop (gfx950): a 256 x 256 tile on 8 waves (two per SIMD), each a
// 64 x 128 piece on v_mfma_f32_32x32x16_bf16; A and B go global -> LDS by
// DMA (global_load_lds_dwordx4) into 5 stages of BK = 32, with the 16-byte
// chunks of each 64-byte row XOR-swizzled by (row >> 2) & 3 so fragment reads
// are conflict free; one barrier per K-step, the refill of K-step kt + 5
// interleaved with the MFMAs of K-step kt.  Tiles are dealt to the 8 XCDs in
// contiguous runs and walked in pairs of M-tiles, N fastest.
#include "sr_device.hpp"

#include <type_traits>

namespace sr {
namespace {

constexpr int BM = 256, BN = 256, BK = 32, THREADS = 512, NS = 5;
constexpr int A_BYTES = BM * 64, B_BYTES = BN * 64, STAGE = A_BYTES + B_BYTES;
constexpr int LPK = 4;   // DMA instructions per wave per K-step (2 A + 2 B blocks of 1 KB)

typedef __attribute__((address_space(3))) char lchar;
typedef unsigned int nu32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 ld16(const lchar* p) {
  return __builtin_bit_cast(uint4, *reinterpret_cast<const __attribute__((address_space(3))) nu32x4*>(p));
}
__device__ __forceinline__ int swz(int r) { return (r >> 2) & 3; }

__device__ __forceinline__ void tile_of(int b, int tm, int tn, int& mt, int& nt) {
  const int nb = tm * tn;
  const int per = nb / 8, rem = nb % 8;
  const int x = b % 8, loc = b / 8;
  const int t = x * per + (x < rem ? x : rem) + loc;
  constexpr int GM = 2;
  const int grp = t / (GM * tn);
  const int first = grp * GM;
  const int gs = (tm - first) < GM ? (tm - first) : GM;
  const int idx = t - grp * GM * tn;
  mt = first + idx % gs;
  nt = idx / gs;
}

__device__ __forceinline__ float silu(float x) { return x * __builtin_amdgcn_rcpf(1.f + __expf(-x)); }

template <int MODE>
__global__ __launch_bounds__(THREADS, 1) void block_gemm_kernel(BlockGemmArgs a, int tiles_m, int tiles_n) {
  if (a.err && *a.err) return;   // the call's table check failed: write nothing
  __shared__ __attribute__((aligned(1024))) char smem_raw[NS * STAGE];
  lchar* smem = (lchar*)smem_raw;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid >> 1, wn = wid & 1;
  const int lc = lane & 31, fhi = lane >> 5;
  int mt, nt;
  tile_of(blockIdx.x, tiles_m, tiles_n, mt, nt);
  const int64_t row0 = (int64_t)mt * BM;
  const int n0 = nt * BN;
  const int K = a.K;
  const int64_t M = a.M;

  // DMA sources: wave wid fills A and B blocks 2 wid, 2 wid + 1 (16 rows each)
  const char* a_src[2];
  const char* b_src[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int row = (wid * 2 + i) * 16 + (lane >> 2);
    const int c = (lane & 3) ^ swz(row);
    int64_t mr = row0 + row;
    mr = mr >= M ? M - 1 : mr;          // rows past M are never stored
    a_src[i] = static_cast<const char*>(a.A) + (mr * K + c * 8) * 2;
    const int n = n0 + row;
    const char* w;
    int64_t wr;
    if constexpr (MODE == kGemmSwiglu) {
      const int blk = row >> 5;          // 32-row blocks alternate gate / up
      wr = (int64_t)nt * 128 + (blk >> 1) * 32 + (row & 31);
      w = static_cast<const char*>((blk & 1) ? a.B2 : a.B);
    } else {
      wr = n;
      w = static_cast<const char*>(a.B);
    }
    b_src[i] = w + (wr * K + c * 8) * 2;
  }
  const int arow = wm * 64 + lc;
  const int brow = wn * 128 + lc;
  const int a_k0 = arow * 64 + ((0 + fhi) ^ swz(arow)) * 16;
  const int a_k1 = arow * 64 + ((2 + fhi) ^ swz(arow)) * 16;
  const int b_k0 = A_BYTES + brow * 64 + ((0 + fhi) ^ swz(brow)) * 16;
  const int b_k1 = A_BYTES + brow * 64 + ((2 + fhi) ^ swz(brow)) * 16;

  bf16x8 fa[2][2], fb[2][4];
  f32x16 acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = zero16();

  // fragment q of a K-step: 0, 1 A (rows +0, +32 of the wave's band), 2..5 B
  auto read_one = [&](int stage, int ks, int slot, int qq) {
    const int q = qq == 0 ? 0 : (qq <= 4 ? qq + 1 : 1);   // order A0, B0..B3, A1
    const lchar* sb = smem + stage * STAGE;
    if (q < 2) fa[slot][q] = as_bf16x8(ld16(sb + (ks ? a_k1 : a_k0) + q * 32 * 64));
    else fb[slot][q - 2] = as_bf16x8(ld16(sb + (ks ? b_k1 : b_k0) + (q - 2) * 32 * 64));
  };
  auto mma_one = [&](int slot, int q) {
    const int i = q >> 2, j = q & 3;
    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[slot][i], fb[slot][j], acc[i][j], 0, 0, 0);
  };
  auto dma_one = [&](int kt, int stage, int q) {
    const uint32_t lds0 = (uint32_t)(uintptr_t)smem + stage * STAGE;
    if (q < 2) dma16(a_src[q] + (int64_t)kt * BK * 2, lds0 + (wid * 2 + q) * 1024);
    else dma16(b_src[q - 2] + (int64_t)kt * BK * 2, lds0 + A_BYTES + (wid * 2 + q - 2) * 1024);
  };

  const int KT = K / BK;
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int q = 0; q < LPK; ++q) dma_one(s < KT ? s : KT - 1, s, q);
  wait_vm<(NS - 1) * LPK>();
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0xc07f);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int q = 0; q < 6; ++q) read_one(0, 0, 0, q);

  int st = 0;
  for (int kt = 0; kt < KT; ++kt) {
    const int st1 = st + 1 == NS ? 0 : st + 1;
    const int kn = kt + NS < KT ? kt + NS : KT - 1;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      mma_one(0, q);
      if (q < 6) read_one(st, 1, 1, q);
      __builtin_amdgcn_sched_barrier(0);
    }
    // this wave's reads of stage st are done and K-step kt + 1 has landed;
    // after the barrier stage st may be refilled and stage st1 read
    wait_vm<(NS - 2) * LPK>();
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      mma_one(1, q);
      if (q < 6) read_one(st1, 0, 0, q);
      if ((q & 1) == 0) dma_one(kn, st, q >> 1);
      __builtin_amdgcn_sched_barrier(0);
    }
    st = st1;
  }
  __builtin_amdgcn_sched_barrier(0);
  wait_vm<0>();                          // no DMA may still be landing in LDS
  __builtin_amdgcn_s_waitcnt(0xc07f);
  __builtin_amdgcn_s_barrier();

  // ---- epilogue: acc[i][j] register r of lane l is tile row
  // 64 wm + 32 i + acc_row(r, l), column 128 wn + 32 j + l % 32
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t row = row0 + wm * 64 + 32 * i + acc_row(r, lane);
      if (row >= M) continue;
      if constexpr (MODE == kGemmSwiglu) {
        uint16_t* out = static_cast<uint16_t*>(a.C) + row * a.ldc + (int64_t)nt * 128 + wn * 64 + lc;
        out[0] = f32_to_bf16_bits(silu(acc[i][0][r]) * acc[i][1][r]);
        out[32] = f32_to_bf16_bits(silu(acc[i][2][r]) * acc[i][3][r]);
      } else {
        float* out = static_cast<float*>(a.C) + row * a.ldc + n0 + wn * 128 + lc;
#pragma unroll
        for (int j = 0; j < 4; ++j) out[32 * j] += acc[i][j][r];
      }
    }
  }
}

template <int MODE>
hipError_t run_gemm(const BlockGemmArgs& a, hipStream_t s) {
  if (a.M == 0) return hipSuccess;
  if (a.K % BK || a.N % BN) return hipErrorInvalidValue;
  const int tm = (int)((a.M + BM - 1) / BM), tn = a.N / BN;
  hipLaunchKernelGGL((block_gemm_kernel<MODE>), dim3(tm * tn), dim3(THREADS), 0, s, a, tm, tn);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_block_gemm(int mode, const BlockGemmArgs& a, hipStream_t s) {
  if (mode == kGemmResid) return run_gemm<kGemmResid>(a, s);
  if (mode == kGemmSwiglu) return run_gemm<kGemmSwiglu>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace sr
