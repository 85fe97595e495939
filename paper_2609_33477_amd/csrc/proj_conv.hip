// Projection GEMM fused with the short causal conv, SiLU, key L2 norm, the
// decay / erase gates and the k | v conv tail (bf16 anchors; bf16 or fp8
// weights).
//
// What it computes (Section 2.1: the update's key, value and gates are linear
// maps of the layer input; Appendix A: a width-w depthwise conv over the q, k, v
// projections whose state is the last w-1 inputs):
//   P      = X [W_k; W_v; W_a; W_b]^T                       (fp32 accumulate)
//   k, v   = SiLU(sum_i cw[c][i] P[t-w+1+i][c])             (zero before the segment start)
//   k_hat  = k / sqrt(|k|^2 + eps)                           (per key head)
//   G      = log2 alpha = -exp(A_log) softplus(a + dt_bias) log2(e)
//   beta   = sigmoid(b)
// The projection never reaches HBM: each 256 x 256 output tile is finished in
// LDS and only k_hat / v (bf16, head-major [H][T][d]), G and beta ([H_v][T],
// fp32) and the tail rows are written.
//
// Main loop (gfx950): 8 waves (two per SIMD), each a 64 x 128 piece of the
// tile on v_mfma_f32_32x32x16_bf16 with fp32 accumulators.  A and B stream
// global -> LDS with global_load_lds_dwordx4 (no register staging) into LDS
// stages of BK = 32 (5 for bf16, 6 for fp8 weights), up to five K-steps ahead
// of the MFMAs; 16-byte chunks are XOR-swizzled inside each 64-byte row so
// fragment reads are conflict free.
// fp8 (E4M3) weights are staged as bytes and converted to bf16 after the
// fragment read (exact); the per-channel scale is folded into the conv taps
// (the conv is linear per column) and applied to the gate and tail values.
// Weights are the MFMA's first operand, so each lane's accumulators hold 4
// consecutive columns of one output row.
// Tiles are dealt in contiguous runs per XCD and walked in groups of 8
// M-tiles so concurrently running tiles share A and B panels in L2.  In a
// narrow last N-tile (the 2 H_v gate columns) waves skip the MFMAs and
// fragment reads of columns past N.
//
// Conv epilogue: M-tiles overlap by 3 rows (stride 253), so every output row's
// w-1 predecessors are in the tile.  Each 128-column half of the accumulator
// tile goes to LDS row-major with 16-byte writes, in 8 bands of 32 rows (one
// per wave) that each also hold a copy of the 3 rows before them.  Lanes l
// and l+32 then own one row, 64 columns each, and walk them 4 at a time:
// conv over the row and the 3 before it, SiLU, and for a key head the sum of
// squares (the two lanes' partial sums combined), with the activation written
// back in place (only these lanes read the row's columns after that) and
// scaled by the inverse norm on a second pass; the outputs leave as 16-byte
// stores.  The segment info and conv taps the epilogue needs are loaded
// before the main loop.
#include "sr_device.hpp"

#include <type_traits>

namespace sr {
namespace {

constexpr int BM = 256, BN = 256, BK = 32, THREADS = 512, WAVES = THREADS / 64;
constexpr int HALO = 3, SM = BM - HALO;           // tile row stride
// Epilogue tile in LDS: one 128-column half of the accumulator tile,
// row-major (pitch EROW floats: 16-byte reads by 16 consecutive rows are
// conflict free), split into 8 bands of 32 rows (one per wave).  Each band
// holds its rows at slots 4..35 and copies of the 3 rows before it at slots
// 1..3, so a lane reads its row and the w-1 rows before it at fixed offsets
// and may overwrite its own row without racing a neighbouring wave.
constexpr int EROW = 132;
constexpr int EBAND = 36;
constexpr int E_BYTES = WAVES * EBAND * EROW * 4;
constexpr int TAP_BYTES = 4 * 128 * 4;              // taps [rows back][column] of one half
constexpr float kLog2e = 1.4426950408889634f;

typedef __attribute__((address_space(3))) char lchar;
typedef __attribute__((address_space(3))) float lfloat;
typedef unsigned int nu32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int nu32x2 __attribute__((ext_vector_type(2)));
typedef float nf32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 ld16(const lchar* p) {
  return __builtin_bit_cast(uint4, *reinterpret_cast<const __attribute__((address_space(3))) nu32x4*>(p));
}
__device__ __forceinline__ uint2 ld8(const lchar* p) {
  return __builtin_bit_cast(uint2, *reinterpret_cast<const __attribute__((address_space(3))) nu32x2*>(p));
}

template <typename TB> struct BT;
// B row bytes per K-step, 1 KB DMA blocks per wave and K-step, LDS stages
// (as many as fit in 160 KB: the deeper the prefetch, the more memory latency
// it hides)
template <> struct BT<bf16_t> { static constexpr int ROW = 64, BLKS = 2, NS = 5; };
template <> struct BT<fp8_t> { static constexpr int ROW = 32, BLKS = 1, NS = 6; };

// 16 bytes per lane, global -> LDS at lds_base + 16 * lane (wave-uniform
// base).  Inline asm: the compiler would otherwise wait for every such load
// before any later LDS read; completion is tracked by hand (wait_vm) before
// the barrier that publishes a stage.
// `lds_off` must be wave-uniform (it is an SGPR operand).
__device__ __forceinline__ void dma16(const void* src, uint32_t lds_off) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds_off), "v"(src) : "memory", "m0");
}

// s_waitcnt vmcnt(N) with lgkmcnt and expcnt left at their maxima
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// 16-byte chunk swizzle inside a 64-byte LDS row.  A fragment read has lanes
// 0-31 on 32 consecutive rows (lanes 32-63 on the next chunk); with this XOR
// every ds_read_b128 is conflict free (measured: 4 LDS cycles per read, the
// 256 B/clk peak), where rows 4 apart must land in different chunks.
__device__ __forceinline__ int swz(int r) { return (r >> 2) & 3; }

// hardware block id -> (m tile, n tile): contiguous runs per XCD (blocks are
// dealt round-robin to the 8 XCDs), then groups of 8 m-tiles walked n-major
__device__ __forceinline__ void tile_of(int b, int tm, int tn, int& mt, int& nt) {
  const int nb = tm * tn;
  const int per = nb / 8, rem = nb % 8;
  const int x = b % 8, loc = b / 8;
  const int t = x * per + (x < rem ? x : rem) + loc;
  constexpr int GM = 8;
  const int grp = t / (GM * tn);
  const int first = grp * GM;
  const int gs = (tm - first) < GM ? (tm - first) : GM;
  const int idx = t - grp * GM * tn;
  mt = first + idx % gs;
  nt = idx / gs;
}


__device__ __forceinline__ void st_f4(lfloat* p, float x, float y, float z, float w) {
  *reinterpret_cast<__attribute__((address_space(3))) nf32x4*>(p) = nf32x4{x, y, z, w};
}

// bf16 scale of fp8 weight column n (selected without branches, one load)
__device__ __forceinline__ const uint16_t* col_scale_ptr(const ProjConvArgs& a, int n) {
  const uint16_t* p = static_cast<const uint16_t*>(a.seg[0].scale) + (n - a.seg[0].n0);
#pragma unroll
  for (int s = 1; s < 4; ++s)
    if (s < a.n_wseg && n >= a.seg[s].n0 && n < a.seg[s].n1) p = static_cast<const uint16_t*>(a.seg[s].scale) + (n - a.seg[s].n0);
  return p;
}
// per-output-column scale of fp8 weights (1 for bf16 weights)
template <typename TB>
__device__ __forceinline__ float col_scale(const ProjConvArgs& a, int n) {
  if constexpr (std::is_same<TB, fp8_t>::value) return bf16_bits_to_f32(*col_scale_ptr(a, n));
  return 1.f;
}

__device__ __forceinline__ float fast_sigmoid(float x) { return __builtin_amdgcn_rcpf(1.f + __expf(-x)); }
__device__ __forceinline__ float softplus(float x) { return fmaxf(x, 0.f) + log1pf(__expf(-fabsf(x))); }

__device__ __forceinline__ float load_elem(const void* p, int64_t i, bool is_bf16) {
  return is_bf16 ? bf16_bits_to_f32(static_cast<const uint16_t*>(p)[i]) : static_cast<const float*>(p)[i];
}
__device__ __forceinline__ void store_elem(void* p, int64_t i, float v, bool is_bf16) {
  if (is_bf16) static_cast<uint16_t*>(p)[i] = f32_to_bf16_bits(v);
  else static_cast<float*>(p)[i] = v;
}

template <typename TB, int D>
__global__ __launch_bounds__(THREADS, 1) void proj_conv_kernel(ProjConvArgs a, int tiles_m, int tiles_n) {
  constexpr int BROW = BT<TB>::ROW, BBLK = BT<TB>::BLKS, NS = BT<TB>::NS;
  constexpr int A_BYTES = BM * 64, B_BYTES = BN * BROW, STAGE = A_BYTES + B_BYTES;
  constexpr int LPK = 2 + BBLK;  // DMA instructions per wave per K-step
  constexpr int LDS = NS * STAGE > E_BYTES + TAP_BYTES ? NS * STAGE : E_BYTES + TAP_BYTES;
  __shared__ __attribute__((aligned(1024))) char smem_raw[LDS];
  lchar* smem = (lchar*)smem_raw;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
  const int wm = wid >> 1, wn = wid & 1;                       // 64-row x 128-column sub-tile
  int mt, nt;
  tile_of(blockIdx.x, tiles_m, tiles_n, mt, nt);
  const int64_t row0 = (int64_t)mt * SM - HALO;  // tile row 0 (negative for the first tile)
  const int n0 = nt * BN;
  const int K = a.K;
  const int64_t T = a.T;

  // Epilogue inputs, fetched before the first DMA so their latency hides
  // under the main loop (and no wait_vm count below has to include them):
  // the segment info of the tile row this lane will own (lanes l and l+32
  // share a row), and the conv tap (fp8 column scale folded in) this thread
  // stages for each half.
  const int lr = lane & 31, ch = lane >> 5;
  const int r = wid * 32 + lr;                // tile row owned by this lane
  const int64_t m = row0 + r;
  RowInfo ri = {0, 0, -1, 0};
  if (m >= 0 && m < T) ri = a.info[m];
  // Raw tap bits: nothing reads them before the epilogue, so no wait for
  // these loads is placed ahead of the main loop.
  uint32_t tap_bits[2] = {0u, 0u};
  uint32_t tap_sc[2] = {0x3f80u, 0x3f80u};   // bf16 bits of the column scale
  {
    const int c = tid >> 2, j = tid & 3;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int n = n0 + h * 128 + c;
      if (n < a.C_kv) {
        if constexpr (std::is_same<TB, fp8_t>::value) tap_sc[h] = *col_scale_ptr(a, n);
        const int64_t i = (int64_t)n * a.w + a.w - 1 - j;
        if (j <= a.w - 1) {
          if (a.conv_bf16) tap_bits[h] = static_cast<const uint16_t*>(a.conv_w)[i];
          else tap_bits[h] = static_cast<const uint32_t*>(a.conv_w)[i];
        }
      }
    }
  }

  // ------------------------------------------------------------ main loop
  // DMA sources: wave wid fills A blocks 2 wid, 2 wid + 1 (16 rows each)
  const char* a_src[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int row = (wid * 2 + i) * 16 + (lane >> 2);
    const int c = (lane & 3) ^ swz(row);
    int64_t mr = row0 + row;
    mr = mr < 0 ? 0 : (mr >= T ? T - 1 : mr);   // rows outside [0, T) are never output
    a_src[i] = static_cast<const char*>(a.A) + (mr * K + c * 8) * 2;
  }
  const char* b_src[BBLK];
#pragma unroll
  for (int i = 0; i < BBLK; ++i) {
    int row, coff;
    if (std::is_same<TB, bf16_t>::value) {
      row = (wid * 2 + i) * 16 + (lane >> 2);
      coff = ((lane & 3) ^ swz(row)) * 8;   // elements
    } else {
      row = wid * 32 + (lane >> 1);
      coff = (lane & 1) * 16;
    }
    const int n = (n0 + row < a.N) ? n0 + row : a.N - 1;
    const char* p = static_cast<const char*>(a.seg[0].ptr);
#pragma unroll
    for (int s = 0; s < 4; ++s)
      if (s < a.n_wseg && n >= a.seg[s].n0 && n < a.seg[s].n1)
        p = static_cast<const char*>(a.seg[s].ptr) + ((int64_t)(n - a.seg[s].n0) * K + coff) * Elem<TB>::bytes;
    b_src[i] = p;
  }

  const int fl = swz(lane & 31), hi = lane >> 5;
  const int a_row_off = (wm * 64 + (lane & 31)) * 64;
  const int a_k0 = a_row_off + ((0 + hi) ^ fl) * 16;
  const int a_k1 = a_row_off + ((2 + hi) ^ fl) * 16;
  int b_k0, b_k1;
  if (std::is_same<TB, bf16_t>::value) {
    const int b_row_off = A_BYTES + (wn * 128 + (lane & 31)) * 64;
    b_k0 = b_row_off + ((0 + hi) ^ fl) * 16;
    b_k1 = b_row_off + ((2 + hi) ^ fl) * 16;
  } else {
    const int b_row_off = A_BYTES + (wn * 128 + (lane & 31)) * 32;
    b_k0 = b_row_off + hi * 8;
    b_k1 = b_row_off + 16 + hi * 8;
  }

  bf16x8 fa[2][2], fb[2][4];
  f32x16 acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = zero16();

  // read order A0, B0, B1, B2, B3, A1: the first MFMAs of a sub-step
  // (A0 x B0..B3) need only the first five reads
  auto read_one = [&](int stage, int ks, int slot, int qq) {
    const int q = qq == 0 ? 0 : (qq <= 4 ? qq + 1 : 1);   // 0,1: A fragments; 2..5: B fragments
    const lchar* sb = smem + stage * STAGE;
    if (q < 2) {
      fa[slot][q] = as_bf16x8(ld16(sb + (ks ? a_k1 : a_k0) + q * 32 * 64));
    } else if (std::is_same<TB, bf16_t>::value) {
      fb[slot][q - 2] = as_bf16x8(ld16(sb + (ks ? b_k1 : b_k0) + (q - 2) * 32 * 64));
    } else {
      const uint2 v = ld8(sb + (ks ? b_k1 : b_k0) + (q - 2) * 32 * 32);
      uint4 o;
      o.x = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(v.x, 1.0f, false));
      o.y = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(v.x, 1.0f, true));
      o.z = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(v.y, 1.0f, false));
      o.w = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(v.y, 1.0f, true));
      fb[slot][q - 2] = as_bf16x8(o);
    }
  };
  // Weights go in as the MFMA's first operand, so acc[i][j] is the
  // transposed 32x32 block: lane l holds row 32 i + l%32 of the wave's
  // sub-tile, columns 32 j + 8 q + 4 (l/32) .. +3 in registers 4q .. 4q+3.
  auto mma_one = [&](int slot, int q) {
    const int i = q >> 2, j = q & 3;
    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[slot][j], fa[slot][i], acc[i][j], 0, 0, 0);
  };
  auto dma_one = [&](int kt, int stage, int q) {
    const uint32_t lds0 = (uint32_t)(uintptr_t)smem + stage * STAGE;
    if (q < 2) dma16(a_src[q] + (int64_t)kt * BK * 2, lds0 + (wid * 2 + q) * 1024);
    else if (q - 2 < BBLK)
      dma16(b_src[q - 2] + (int64_t)kt * BK * Elem<TB>::bytes, lds0 + A_BYTES + (wid * BBLK + q - 2) * 1024);
  };

  // The main loop, specialised on the number NJ of 32-column B fragments
  // this wave multiplies: 4, or fewer in the narrow last N-tile (for the
  // shapes here: the gate columns), where waves skip the MFMAs and fragment
  // reads of columns past N but keep the DMA share and every barrier.
  auto main_loop = [&](auto nj_tag) {
    constexpr int NJ = decltype(nj_tag)::value;
    auto read_used = [&](int qq) { return qq == 0 || qq > 4 || qq - 1 < NJ; };
    const int KT = K / BK;
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int q = 0; q < LPK; ++q) dma_one(s < KT ? s : KT - 1, s, q);
    wait_vm<(NS - 1) * LPK>();
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0xc07f);   // no scalar loads in flight at loop entry
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int q = 0; q < 6; ++q) if (read_used(q)) read_one(0, 0, 0, q);

    int st = 0;                              // stage of K-step kt
    for (int kt = 0; kt < KT; ++kt) {
      const int st1 = st + 1 == NS ? 0 : st + 1;
      const int kn = kt + NS < KT ? kt + NS : KT - 1;
      // MFMAs 0-7 (first k16, slot 0) with the second k16's fragments into
      // slot 1 over the first 6
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        if ((q & 3) < NJ) mma_one(0, q);
        if (q < 6 && read_used(q)) read_one(st, 1, 1, q);
        __builtin_amdgcn_sched_barrier(0);
      }
      // Hand-over: this wave's reads of stage st are complete and its loads of
      // K-step kt+1 have landed; after the barrier that holds for every wave,
      // so stage st can be refilled and stage st1 read.
      wait_vm<(NS - 2) * LPK>();
      __builtin_amdgcn_s_waitcnt(0xc07f);
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      // MFMAs 8-15 (slot 1): the next K-step's first fragments into slot 0
      // over the first 6, one refill load every other MFMA (K-step kt+NS,
      // clamped: the surplus refills of the last steps land in stages nobody
      // reads again)
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        if ((q & 3) < NJ) mma_one(1, q);
        if (q < 6 && read_used(q)) read_one(st1, 0, 0, q);
        if ((q & 1) == 0 && (q >> 1) < LPK) dma_one(kn, st, q >> 1);
        __builtin_amdgcn_sched_barrier(0);
      }
      st = st1;
    }
  };
  const int n_wave = a.N - (n0 + wn * 128);        // valid columns of this wave's 128
  if (n_wave > 64) main_loop(std::integral_constant<int, 4>{});
  else if (n_wave > 0) main_loop(std::integral_constant<int, 2>{});
  else main_loop(std::integral_constant<int, 0>{});
  __builtin_amdgcn_sched_barrier(0);
  wait_vm<0>();                      // no DMA may land in LDS once it is reused
  __builtin_amdgcn_s_waitcnt(0xc07f);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);

  // ------------------------------------------------------------ epilogue
  // Lanes l and l+32 own tile row 32 wid + l%32; lane half ch handles
  // columns [64 ch, 64 ch + 64) of each 128-column half.
  constexpr int CW = D < 64 ? D : 64;          // columns of one head a lane handles
  constexpr int HPL = 64 / CW;                 // heads (or head halves) per lane
  lfloat* E = (lfloat*)smem_raw;
  lfloat* TAPS = (lfloat*)(smem_raw + E_BYTES);
  lfloat* erow = E + (wid * EBAND + 4 + lr) * EROW;   // slot of row r
  const bool out = r >= HALO && m < T;        // m >= 0 holds for r >= HALO
  const bool need_mask = __builtin_amdgcn_ballot_w64(out && ri.pos < HALO) != 0;
  const int w1 = a.w - 1;
  const bool tail_row = a.tail != nullptr && out && ri.slot >= 0 && ri.rem <= w1;
  const bool any_tail = __builtin_amdgcn_ballot_w64(tail_row) != 0;
  const bool tail_bf16 = a.tail_bf16 != 0;

  for (int h = 0; h < 2; ++h) {
    const int nh0 = n0 + h * 128;
    if (nh0 >= a.N) break;
    if (h) {
      __builtin_amdgcn_s_waitcnt(0xc07f);
      __builtin_amdgcn_s_barrier();     // every wave is done reading half 0
    }
    if (wn == h) {
      // 16-byte row-major writes (4 consecutive columns per lane); 16 rows
      // 132 floats apart cover all 64 banks once
      const int c4 = 4 * (lane >> 5);
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int band = wm * 2 + i;
        lfloat* dst = E + (band * EBAND + 4 + lr) * EROW + c4;
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            st_f4(dst + j * 32 + 8 * q, acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
        // the last 3 rows of a band are also the next band's halo
        if (band < WAVES - 1 && lr >= 29) {
          lfloat* hdst = E + ((band + 1) * EBAND + 1 + (lr - 29)) * EROW + c4;
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q)
              st_f4(hdst + j * 32 + 8 * q, acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
        }
      }
    }
    {
      // conv taps of this half's k | v columns: TAPS[j][c] multiplies row t-j
      // (an fp8 column's scale is folded in: the conv is linear per column)
      const int c = tid >> 2, j = tid & 3;
      const float sc = bf16_bits_to_f32((uint16_t)(h ? tap_sc[1] : tap_sc[0]));
      const int sh = a.conv_bf16 ? 16 : 0;
      TAPS[j * 128 + c] = __builtin_bit_cast(float, (h ? tap_bits[1] : tap_bits[0]) << sh) * sc;
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_s_barrier();

    for (int hl = 0; hl < HPL; ++hl) {
      const int c0 = 64 * ch + hl * CW;       // first column of this lane's piece, in the half
      const int e0 = c0 % D;                  // its offset inside the head
      const int nb = nh0 + c0 - e0;           // first projection column of the head
      if (nb >= a.N) continue;
      if (nb < a.C_kv) {
        // ---- k or v head: conv, SiLU, (key) L2 norm.  Columns go 4 at a
        // time (16-byte reads of this row and the 3 before it).
        const bool is_k = nb < a.C_k;
        const int hh = is_k ? nb / D : (nb - a.C_k) / D;
        auto conv4 = [&](int c, auto mask_tag) {
          constexpr bool MASK = decltype(mask_tag)::value;
          nf32x4 x[4], tp[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            x[j] = *reinterpret_cast<const __attribute__((address_space(3))) nf32x4*>(erow - j * EROW + c);
            tp[j] = *reinterpret_cast<const __attribute__((address_space(3))) nf32x4*>(TAPS + j * 128 + c);
          }
          if (MASK) {
#pragma unroll
            for (int j = 1; j < 4; ++j)
              if (ri.pos < j) x[j] = nf32x4{0.f, 0.f, 0.f, 0.f};
          }
          nf32x4 y;
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            float v = tp[0][u] * x[0][u];
            v = fmaf(tp[1][u], x[1][u], v);
            v = fmaf(tp[2][u], x[2][u], v);
            v = fmaf(tp[3][u], x[3][u], v);
            y[u] = v * fast_sigmoid(v);
          }
          return y;
        };
        char* dst = static_cast<char*>(is_k ? a.Kbuf : a.Vbuf) + (((int64_t)hh * T + (out ? m : 0)) * D + e0) * 2;
        auto head_pass = [&](auto mask_tag) {
          // pass 1: y and (keys) its sum of squares; y replaces x in this
          // row's slot (rows after it have read x already: same wave,
          // earlier instruction; the next band reads its own halo copy)
          float ss0 = 0.f, ss1 = 0.f;
          __builtin_amdgcn_s_waitcnt(0xc07f);
#pragma unroll 4
          for (int c = c0; c < c0 + CW; c += 4) {
            const nf32x4 y = conv4(c, mask_tag);
            ss0 = fmaf(y[0], y[0], fmaf(y[1], y[1], ss0));
            ss1 = fmaf(y[2], y[2], fmaf(y[3], y[3], ss1));
            *reinterpret_cast<__attribute__((address_space(3))) nf32x4*>(erow + c) = y;
          }
          float ss = ss0 + ss1;
          if constexpr (D > 64) {
            // the other 64 columns of the head are in lane l ^ 32
            ss += __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute((lane ^ 32) << 2, __builtin_bit_cast(int, ss)));
          }
          const float inv = is_k ? 1.f / sqrtf(ss + a.eps) : 1.f;
#pragma unroll 4
          for (int q = 0; q < CW / 8; ++q) {
            const nf32x4 y0 = *reinterpret_cast<const __attribute__((address_space(3))) nf32x4*>(erow + c0 + 8 * q);
            const nf32x4 y1 = *reinterpret_cast<const __attribute__((address_space(3))) nf32x4*>(erow + c0 + 8 * q + 4);
            uint4 o;
            o.x = pack_bf16x2(y0[0] * inv, y0[1] * inv);
            o.y = pack_bf16x2(y0[2] * inv, y0[3] * inv);
            o.z = pack_bf16x2(y1[0] * inv, y1[1] * inv);
            o.w = pack_bf16x2(y1[2] * inv, y1[3] * inv);
            if (out) *reinterpret_cast<uint4*>(dst + q * 16) = o;
          }
        };
        // the raw projection of the segment's last w-1 rows is the conv state
        // (before the pass overwrites the row)
        if (any_tail && tail_row) {
          for (int e = 0; e < CW; ++e)
            store_elem(a.tail, ((int64_t)ri.slot * a.c_tail + a.tail_kv_off + nb + e0 + e) * w1 + (w1 - ri.rem),
                       erow[c0 + e] * col_scale<TB>(a, nb + e0 + e), tail_bf16);
        }
        if (need_mask) head_pass(std::true_type{});
        else head_pass(std::false_type{});
      } else {
        // ---- gate columns: G = log2 alpha from a, beta from b (no conv)
        for (int e = 0; e < CW; ++e) {
          const int n = nb + e0 + e;
          if (n >= a.N) break;
          const float x = erow[c0 + e] * col_scale<TB>(a, n);
          if (n < a.C_kv + a.H_v) {
            const int hv = n - a.C_kv;
            const float gl = -__expf(a.a_log[hv]) * softplus(x + a.dt_bias[hv]) * kLog2e;
            if (out) a.Gbuf[(int64_t)hv * T + m] = gl;
          } else {
            const int hv = n - a.C_kv - a.H_v;
            if (out) a.Bbuf[(int64_t)hv * T + m] = fast_sigmoid(x);
          }
        }
      }
    }
  }
}

template <typename TB, int D>
hipError_t run(const ProjConvArgs& a, hipStream_t s) {
  if (a.T == 0) return hipSuccess;
  if (a.K % BK) return hipErrorInvalidValue;
  const int tm = (int)((a.T + SM - 1) / SM), tn = (a.N + BN - 1) / BN;
  hipLaunchKernelGGL((proj_conv_kernel<TB, D>), dim3(tm * tn), dim3(THREADS), 0, s, a, tm, tn);
  return hipGetLastError();
}

template <typename TB>
hipError_t by_head(int d, const ProjConvArgs& a, hipStream_t s) {
  switch (d) {
    case 32: return run<TB, 32>(a, s);
    case 64: return run<TB, 64>(a, s);
    case 128: return run<TB, 128>(a, s);
  }
  return hipErrorInvalidValue;
}

// One block per segment: position in the segment, rows left, slot.
__global__ void row_info_kernel(const int32_t* cu, const int32_t* slot_ids, RowInfo* info) {
  const int b = blockIdx.x;
  const int32_t s0 = cu[b], s1 = cu[b + 1];
  const int32_t slot = slot_ids ? slot_ids[b] : b;
  for (int32_t t = s0 + (int32_t)threadIdx.x; t < s1; t += (int32_t)blockDim.x) {
    RowInfo v;
    v.pos = t - s0;
    v.rem = s1 - t;
    v.slot = slot;
    v.seg = b;
    info[t] = v;
  }
}

}  // namespace

hipError_t launch_row_info(const int32_t* cu, const int32_t* slot_ids, int32_t n_seg, RowInfo* info,
                           hipStream_t s) {
  if (n_seg == 0) return hipSuccess;
  hipLaunchKernelGGL(row_info_kernel, dim3(n_seg), dim3(256), 0, s, cu, slot_ids, info);
  return hipGetLastError();
}

hipError_t launch_proj_conv(int weight_dtype, int d_head, const ProjConvArgs& a, hipStream_t s) {
  if (weight_dtype == SR_BF16) return by_head<bf16_t>(d_head, a, s);
  if (weight_dtype == SR_FP8_E4M3) return by_head<fp8_t>(d_head, a, s);
  return hipErrorInvalidValue;
}

}  // namespace sr
