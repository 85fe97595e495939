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
// registers and only k_hat / v (bf16, head-major [H][T][d]), G and beta ([H_v][T],
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
// Anchors are the MFMA's first operand and their rows are fed in the order
// that leaves each lane's accumulators holding 32 consecutive rows of one
// column (tok_row).
// Tiles are dealt in contiguous runs per XCD and walked in pairs of M-tiles
// (N-tiles fastest), so the 32 tiles an XCD runs at once span about 2
// anchor panels and 16 weight panels, each fetched into its L2 once for
// many tiles (of group sizes 1 to 32, 2 measured fastest).  In a
// narrow last N-tile (the 2 H_v gate columns) waves skip the MFMAs and
// fragment reads of columns past N.
//
// Rectangular heads (RECT: OLMo-Hybrid's 96-wide keys and 192-wide values,
// Appendix A): each key head takes 128 output columns, its last 32 computed
// from a repeated weight row and zeroed before the conv, so the per-wave key
// norm is unchanged; keys stay in that padded layout, each value head is
// stored as two 96-column halves padded the same way (the scan runs them as
// two square units of 128), and every channel index into the caller's
// weights, scales, conv taps and tail goes through real_col.  The pad costs a tenth
// more MFMA work at OLMo's shape, against an unfused projection whose fp32
// rows went through HBM.
//
// Conv epilogue, in registers: M-tiles overlap by 3 rows (stride 253), so
// every output row's w-1 predecessors are in the tile.  Lane l of wave w
// holds rows 64 (w / 2) + 32 (l / 32) + 0..31 of 4 columns; the conv runs
// down those registers (the 3 rows above the lane's first come from the
// lane before it through a small LDS exchange), then SiLU, in place.  A
// key's sum of squares over its head's columns is summed over the lane's
// blocks and then across the 32 lanes of the half-wave by a DPP
// reduce-scatter; the inverse norms go back to the lanes through the LDS.
// Outputs leave as bf16 pairs (two rows per pack).  Rows near a segment
// start, a segment end (the conv tail) or the tile edge take masked
// variants decided per row for the whole wave.  The segment info and conv
// taps the epilogue needs are loaded before the main loop.
//
// Gate columns (no conv) leave through a per-wave LDS transpose, so their
// head-major G and beta planes get stores of 64 consecutive rows of a head.
//
// One launch covers up to kProjBatch layers of a call (same T and N): the
// grid holds the tiles of all of them, their m-tiles stacked for the walk
// above, and each block reads its layer's arguments from the kernel
// argument segment.  Blocks past the tiles compute the q part of the conv
// tail and the tail's leading zeros (tail_q.hpp): they need nothing the
// tiles write, so they run in the grid's last, partial round or on CUs the
// tiles leave idle.
#include "sr_device.hpp"
#include "tail_q.hpp"

#include <cstddef>
#include <type_traits>
#include <utility>

namespace sr {
namespace {

constexpr int BM = 256, BN = 256, BK = 32, THREADS = 512, WAVES = THREADS / 64;
constexpr int HALO = 3, SM = BM - HALO;           // tile row stride
// Epilogue exchange area (in the last main-loop stage): the last 3 rows of
// each lane's 4 columns, and the inverse key norms of each half-wave's rows.
constexpr int XB_BYTES = WAVES * 64 * 12 * 4;
constexpr int INV_BYTES = WAVES * 2 * 4 * 32 * 4;
constexpr int EPI_BYTES = XB_BYTES + INV_BYTES;
// Gate columns go through the LDS (below the exchange area) so that one store
// covers 64 consecutive rows of a head: per wave a 32-column block, column
// pitch 68 floats (17 x 16 bytes: the 16-byte writes of 16 lanes fall on
// distinct bank groups).
constexpr int GATE_PITCH = 68;
constexpr int GATE_BYTES = WAVES * 32 * GATE_PITCH * 4;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

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

// 16-byte chunk swizzles inside a 64-byte LDS row.  A fragment read is
// serviced 16 lanes at a time; rows r and r + 4 share a bank quarter, so the
// 4 rows of each quarter a 16-lane group reads must sit in distinct chunks
// (measured: 4 LDS cycles per ds_read_b128, the 256 B/clk peak).  Weight
// fragments read 16 consecutive rows; anchor fragments read rows in the
// order of tok_row, whose bank-quarter mates differ in bits 2 and 5.
__device__ __forceinline__ int swz_b(int r) { return (r >> 2) & 3; }
__device__ __forceinline__ int swz_a(int r) { return ((r >> 2) & 1) | ((r >> 4) & 2); }

// Anchor row (within a wave's 64-row band, block 0; block 1 adds 16) fed to
// MFMA row m.  The 32x32 accumulator puts MFMA row 8 (r / 4) + 4 (l / 32) +
// r % 4 in register r of lane l, so with this order lane l holds rows
// 32 (l / 32) + r: 32 consecutive rows per lane over the two blocks, which
// lets the conv run down a lane's own registers.
__device__ __forceinline__ int tok_row(int m) { return 32 * ((m >> 2) & 1) + 4 * (m >> 3) + (m & 3); }

// One step of a reduce-scatter over the 32 lanes of a half-wave: lanes whose
// bit BIT is b keep half b of the N values and add the partner's copy of it
// (partner: a lane with bit BIT flipped and bits below it equal; DPP control
// CTRL, or ds_swizzle xor 16 when CTRL < 0).
template <int N, int BIT, int CTRL>
__device__ __forceinline__ void bfly_step(float* s, int lc) {
  const bool b = (lc >> BIT) & 1;
#pragma unroll
  for (int i = 0; i < N / 2; ++i) {
    const float lo = s[i], hi = s[i + N / 2];
    const float send = b ? lo : hi, keep = b ? hi : lo;
    int r;
    if constexpr (CTRL < 0) r = __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, send), 0x401F);
    else r = __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, send), CTRL, 0xF, 0xF, false);
    s[i] = keep + __builtin_bit_cast(float, r);
    if (i % 4 == 3) __builtin_amdgcn_sched_barrier(0);   // bounds the scheduler's interleaving
  }
}

// OR / AND of a 32-bit value over the 64 lanes (the result is wave-uniform)
template <bool OR>
__device__ __forceinline__ uint32_t wave_reduce(uint32_t v) {
  auto op = [](uint32_t x, int y) { return OR ? x | (uint32_t)y : x & (uint32_t)y; };
  v = op(v, __builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false));    // lane ^ 1
  v = op(v, __builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false));    // lane ^ 2
  v = op(v, __builtin_amdgcn_mov_dpp((int)v, 0x124, 0xF, 0xF, false));   // quad g -/+ 1
  v = op(v, __builtin_amdgcn_mov_dpp((int)v, 0x128, 0xF, 0xF, false));   // quads g -/+ 2, 3
  v = op(v, __builtin_amdgcn_ds_swizzle((int)v, 0x401F));                // lane ^ 16
  return op((uint32_t)__builtin_amdgcn_readlane((int)v, 0), __builtin_amdgcn_readlane((int)v, 32));
}

// f(integral_constant<int, i>) for i = 0 .. N-1, unrolled at compile time
// (register arrays indexed by i stay in registers)
template <int N, typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl<N>(f, std::make_integer_sequence<int, N>{});
}

// hardware block id -> (m tile, n tile): contiguous runs per XCD (blocks are
// dealt round-robin to the 8 XCDs), then pairs of m-tiles walked n-major
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


__device__ __forceinline__ void st_f4(lfloat* p, float x, float y, float z, float w) {
  *reinterpret_cast<__attribute__((address_space(3))) nf32x4*>(p) = nf32x4{x, y, z, w};
}

// bf16 scale of fp8 weight column n (selected without branches, one load)
__device__ __forceinline__ const uint16_t* col_scale_ptr(const ProjConvArgs& a, int n) {
  const uint16_t* p = static_cast<const uint16_t*>(a.seg[0].scale) + (n - a.seg[0].n0);
#pragma unroll
  for (int s = 1; s < 6; ++s)
    if (s < a.n_wseg && n >= a.seg[s].n0 && n < a.seg[s].n1) p = static_cast<const uint16_t*>(a.seg[s].scale) + (n - a.seg[s].n0);
  return p;
}
// Output column n -> the caller's channel order (weight rows, fp8 scales,
// conv taps, tail channels).  Square heads: n itself.  RECT: key head h's
// output columns h D + j map to channel h k_real + j (the pad columns
// j >= k_real to the head's last channel: their products are discarded),
// and the value and gate columns shift down by the keys' padding.
template <bool RECT, int D>
__device__ __forceinline__ int real_col(const ProjConvArgs& a, int n) {
  if constexpr (!RECT) return n;
  const int pad = (a.C_k / D) * (D - a.k_real);
  if (n >= a.C_k) return n - pad;
  const int h = n / D, j = n - h * D;
  return h * a.k_real + (j < a.k_real ? j : a.k_real - 1);
}
// per-output-column scale of fp8 weights (1 for bf16 weights)
template <typename TB>
__device__ __forceinline__ float col_scale(const ProjConvArgs& a, int n) {
  if constexpr (std::is_same<TB, fp8_t>::value) return bf16_bits_to_f32(*col_scale_ptr(a, n));
  return 1.f;
}

__device__ __forceinline__ float fast_sigmoid(float x) { return __builtin_amdgcn_rcpf(1.f + __expf(-x)); }
// max(x, 0) + ln(1 + e^-|x|) on the hardware exp and log: where e^-|x| is
// below half an ulp of 1 the second term drops out, an absolute error under
// 6e-8 in a value that then scales a log-decay
__device__ __forceinline__ float softplus(float x) { return fmaxf(x, 0.f) + __logf(1.f + __expf(-fabsf(x))); }

__device__ __forceinline__ float load_elem(const void* p, int64_t i, bool is_bf16) {
  return is_bf16 ? bf16_bits_to_f32(static_cast<const uint16_t*>(p)[i]) : static_cast<const float*>(p)[i];
}
__device__ __forceinline__ void store_elem(void* p, int64_t i, float v, bool is_bf16) {
  if (is_bf16) static_cast<uint16_t*>(p)[i] = f32_to_bf16_bits(v);
  else static_cast<float*>(p)[i] = v;
}

template <typename TB, int D, bool RECT>
__global__ __launch_bounds__(THREADS, 1) void proj_conv_kernel(ProjConvBatch pb, int tiles_m, int tiles_n) {
  // The batch is the kernel's first argument: a layer's arguments are read
  // from the argument segment at a block-uniform offset.
  const char* kargs = (const char*)__builtin_amdgcn_kernarg_segment_ptr();
  auto layer_args = [&](int l) -> const ProjConvArgs& {
    return *reinterpret_cast<const ProjConvArgs*>(kargs + offsetof(ProjConvBatch, layer) + l * sizeof(ProjConvArgs));
  };
  if (pb.layer[0].err && *pb.layer[0].err) return;   // the call's table check failed: write nothing
  constexpr int BROW = BT<TB>::ROW, BBLK = BT<TB>::BLKS, NS = BT<TB>::NS;
  constexpr int A_BYTES = BM * 64, B_BYTES = BN * BROW, STAGE = A_BYTES + B_BYTES;
  constexpr int LPK = 2 + BBLK;  // DMA instructions per wave per K-step
  constexpr int EPI_OFF = (NS - 1) * STAGE;   // epilogue exchange area: the last stage
  constexpr int LDS = NS * STAGE > EPI_OFF + EPI_BYTES ? NS * STAGE : EPI_OFF + EPI_BYTES;
  __shared__ __attribute__((aligned(1024))) char smem_raw[LDS];
  lchar* smem = (lchar*)smem_raw;
  static_assert(LDS >= kTqLds && THREADS == 64 * kTqWaves, "q-tail blocks share the tile's LDS and waves");
  static_assert(GATE_BYTES <= EPI_OFF, "gate transposes below the epilogue exchange area");
  const int n_tiles = pb.n_layers * tiles_m * tiles_n;
  if ((int)blockIdx.x >= n_tiles) {
    const int b = (int)blockIdx.x - n_tiles;
    int l = 0;
    while (l + 1 < pb.n_layers && b >= pb.tq_off[l + 1]) ++l;
    const TailArgs& tq = layer_args(l).tq;
    const int bl = b - pb.tq_off[l], gx = tail_q_grid_x(tq);
    tail_q_block<TB>(tq, bl % gx, bl / gx, smem_raw);
    return;
  }

  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
  const int wm = wid >> 1, wn = wid & 1;                       // 64-row x 128-column sub-tile
  const int hf = lane >> 5, lc = lane & 31;
  // m-tiles of the layers stacked: the XCD-aware walk runs over all of them
  int mt, nt;
  tile_of(blockIdx.x, pb.n_layers * tiles_m, tiles_n, mt, nt);
  const int layer = mt / tiles_m;
  mt -= layer * tiles_m;
  const ProjConvArgs& a = layer_args(layer);
  const int64_t row0 = (int64_t)mt * SM - HALO;  // tile row 0 (negative for the first tile)
  const int n0 = nt * BN;
  const int K = a.K;
  const int64_t T = a.T;

  // The epilogue share of this lane: tile rows rbase .. rbase + 31 of the
  // columns ncol + 32 j (j = 0..3).  Its inputs are fetched before the first
  // DMA so their latency hides under the main loop (and no wait_vm count
  // below has to include them): the segment position and rows left of the
  // first row, the raw conv taps of the four columns and their fp8 scales.
  const int rbase = wm * 64 + 32 * hf;
  const int64_t t0 = row0 + rbase;
  const int ncol = n0 + 128 * wn + lc;
  int pos0 = -1, rem0 = 0;
  if (t0 >= 0 && t0 < T) {
    const int2 pr = *reinterpret_cast<const int2*>(a.info + t0);
    pos0 = pr.x;
    rem0 = pr.y;
  }
  // Raw conv taps, decoded in the epilogue (touching them here would make the
  // prologue wait for the loads): with w = 4 and an aligned table, one 8-byte
  // (bf16) or 16-byte (fp32) load per column, [row t-3, t-2, t-1, t]; else
  // one element per tap, tr[j][d] holding the tap of row t - d.
  const int tap_mode = (a.w == 4 && (reinterpret_cast<uintptr_t>(a.conv_w) & 15) == 0) ? (a.conv_bf16 ? 1 : 2) : 0;
  uint32_t tr[4][4], sc_raw[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int n_out = ncol + 32 * j;
    const int n = real_col<RECT, D>(a, n_out);
    sc_raw[j] = 0x3f80u;   // bf16 bits of 1
#pragma unroll
    for (int d = 0; d < 4; ++d) tr[j][d] = 0u;
    if (n_out < a.N) {
      if constexpr (std::is_same<TB, fp8_t>::value) sc_raw[j] = *col_scale_ptr(a, n);
    }
    if (n_out < a.C_kv) {
      if (tap_mode == 1) {
        const uint2 v = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(a.conv_w) + (int64_t)n * 4);
        tr[j][0] = v.x;
        tr[j][1] = v.y;
      } else if (tap_mode == 2) {
        const uint4 v = *reinterpret_cast<const uint4*>(static_cast<const float*>(a.conv_w) + (int64_t)n * 4);
        tr[j][0] = v.x;
        tr[j][1] = v.y;
        tr[j][2] = v.z;
        tr[j][3] = v.w;
      } else {
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          if (d < a.w) {
            const int64_t i = (int64_t)n * a.w + a.w - 1 - d;   // tap of row t - d
            tr[j][d] = a.conv_bf16 ? (uint32_t) static_cast<const uint16_t*>(a.conv_w)[i]
                                   : static_cast<const uint32_t*>(a.conv_w)[i];
          }
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
    const int c = (lane & 3) ^ swz_a(row);
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
      coff = ((lane & 3) ^ swz_b(row)) * 8;   // elements
    } else {
      row = wid * 32 + (lane >> 1);
      coff = (lane & 1) * 16;
    }
    const int n = real_col<RECT, D>(a, (n0 + row < a.N) ? n0 + row : a.N - 1);
    const char* p = static_cast<const char*>(a.seg[0].ptr);
#pragma unroll
    for (int s = 0; s < 6; ++s)
      if (s < a.n_wseg && n >= a.seg[s].n0 && n < a.seg[s].n1)
        p = static_cast<const char*>(a.seg[s].ptr) + ((int64_t)(n - a.seg[s].n0) * K + coff) * Elem<TB>::bytes;
    b_src[i] = p;
  }

  // A fragment of lane l (MFMA row l % 32 of block i): the anchor row that
  // makes lane l's accumulators rows rbase + 16 i .. + 15 in order (see
  // tok_row)
  const int fhi = lane >> 5;
  const int arow = wm * 64 + tok_row(lc);
  const int a_k0 = arow * 64 + ((0 + fhi) ^ swz_a(arow)) * 16;
  const int a_k1 = arow * 64 + ((2 + fhi) ^ swz_a(arow)) * 16;
  int b_k0, b_k1;
  if (std::is_same<TB, bf16_t>::value) {
    const int brow = wn * 128 + (lane & 31);
    b_k0 = A_BYTES + brow * 64 + ((0 + fhi) ^ swz_b(brow)) * 16;
    b_k1 = A_BYTES + brow * 64 + ((2 + fhi) ^ swz_b(brow)) * 16;
  } else {
    const int b_row_off = A_BYTES + (wn * 128 + (lane & 31)) * 32;
    b_k0 = b_row_off + fhi * 8;
    b_k1 = b_row_off + 16 + fhi * 8;
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
      fa[slot][q] = as_bf16x8(ld16(sb + (ks ? a_k1 : a_k0) + q * 16 * 64));
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
  // Anchors go in as the MFMA's first operand: acc[i][j] register r of lane
  // l is column 32 j + l % 32 of the wave's sub-tile at MFMA row
  // 8 (r / 4) + 4 (l / 32) + r % 4, which tok_row maps to tile row
  // rbase + 16 i + r.
  auto mma_one = [&](int slot, int q) {
    const int i = q >> 2, j = q & 3;
    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[slot][i], fb[slot][j], acc[i][j], 0, 0, 0);
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
  // Lane (hf, lc) holds x = the raw projection of its 4 columns at its 32
  // consecutive tile rows: x(j, u) = acc[u / 16][j][u % 16] is row rbase + u
  // of column ncol + 32 j.  The conv runs down those registers; only the 3
  // rows before rbase come from another lane (lane l ^ 32 of this wave for
  // hf = 1, of the wave above for hf = 0), through the LDS.
#define XU(j, u) acc[(u) >> 4][j][(u) & 15]
  // RECT: a key head's pad columns (its 32-column blocks from k_real on)
  // hold products of a repeated weight row; they enter neither the conv
  // halo, the tail, nor the key's norm
  const bool rect_k = RECT && n0 + 128 * wn < a.C_k;
  if constexpr (RECT) {
    if (rect_k) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (32 * j >= a.k_real)
#pragma unroll
          for (int u = 0; u < 32; ++u) XU(j, u) = 0.f;
    }
  }
  lfloat* XB = (lfloat*)(smem_raw + EPI_OFF);
  lfloat* INV = (lfloat*)(smem_raw + EPI_OFF + XB_BYTES);
  {
    lfloat* p = XB + (wid * 64 + lane) * 12;
    st_f4(p, XU(0, 29), XU(1, 29), XU(2, 29), XU(3, 29));
    st_f4(p + 4, XU(0, 30), XU(1, 30), XU(2, 30), XU(3, 30));
    st_f4(p + 8, XU(0, 31), XU(1, 31), XU(2, 31), XU(3, 31));
  }
  __builtin_amdgcn_s_waitcnt(0xc07f);
  __builtin_amdgcn_s_barrier();
  nf32x4 xp[3];    // xp[k][j]: row rbase - 3 + k of column j (zero above the tile)
  {
    const lfloat* p = XB + ((hf ? wid : (wid >= 2 ? wid - 2 : wid)) * 64 + (lane ^ 32)) * 12;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      xp[k] = *reinterpret_cast<const __attribute__((address_space(3))) nf32x4*>(p + 4 * k);
      if (rbase == 0) xp[k] = nf32x4{0.f, 0.f, 0.f, 0.f};
    }
  }

  const int w1 = a.w - 1;
  // Fast case: all 32 rows lie inside one segment, at least w - 1 rows past
  // its start (or are the tile's first rows, which are not output) and more
  // than w - 1 rows before its end (no tail rows).  Otherwise the masks are
  // built from the rows' segment info.
  const bool fast = rem0 >= 32 + w1 && (pos0 >= w1 || rbase == 0);
  const bool wave_fast = __builtin_amdgcn_ballot_w64(!fast) == 0;
  // bit u of m1 / m2 / m3: row u may use row u-1 / u-2 / u-3 (same segment);
  // outm: row u is an output; tailm: row u is one of its segment's last w-1
  // rows (the conv state)
  uint32_t m1 = ~0u, m2 = ~0u, m3 = ~0u, outm = rbase ? ~0u : ~7u, tailm = 0u;
  if (!wave_fast && !fast) {
    m1 = m2 = m3 = outm = 0u;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      int2 pr[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int64_t t = t0 + 8 * b + k;
        pr[k] = int2{-1, 0};
        if (t >= 0 && t < T) pr[k] = *reinterpret_cast<const int2*>(a.info + t);
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int u = 8 * b + k;
        const uint32_t bit = 1u << u;
        if (pr[k].x >= 1) m1 |= bit;
        if (pr[k].x >= 2) m2 |= bit;
        if (pr[k].x >= 3) m3 |= bit;
        if (pr[k].x >= 0 && rbase + u >= HALO) {
          outm |= bit;
          if (pr[k].y <= w1) tailm |= bit;
        }
      }
    }
  }
  if (a.tail == nullptr) tailm = 0u;
  const bool tail_bf16 = a.tail_bf16 != 0;
  // Wave-uniform row sets: cmask, the rows where some lane masks a conv
  // term; ofull, the rows every lane outputs (rows 0-2 of the tile are not).
  uint32_t cmask = 0u, ofull = wm == 0 ? ~7u : ~0u;
  if (!wave_fast) {
    cmask = wave_reduce<true>(~(m1 & m2 & m3));
    ofull = wave_reduce<false>(outm);
  }
  const bool any_tail = __builtin_amdgcn_ballot_w64(tailm != 0u) != 0;

  // conv taps (row t - d) with the fp8 column scale and -log2(e) folded in:
  // the conv yields z = -log2(e) c, so e^-c = 2^z and SiLU(c) = -ln2 z / (1 + 2^z)
  float tp[4][4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      uint32_t bits;
      if (tap_mode == 1) bits = (d & 1) ? tr[j][(3 - d) >> 1] << 16 : tr[j][(3 - d) >> 1] & 0xffff0000u;
      else if (tap_mode == 2) bits = tr[j][3 - d];
      else bits = a.conv_bf16 ? tr[j][d] << 16 : tr[j][d];
      tp[j][d] = __builtin_bit_cast(float, bits) * bf16_bits_to_f32(sc_raw[j]) * -kLog2e;
    }
  }

  // store of row u: unconditional where every lane outputs it
  auto row_store = [&](auto* p, auto v, int u) {
    if ((ofull >> u) & 1u) *p = v;
    else if ((outm >> u) & 1u) *p = v;
  };

  constexpr int NH = 128 / D, JB = D / 32;   // heads per wave, 32-column blocks per head
  static_for<NH>([&](auto hd_c) {
    constexpr int hd = decltype(hd_c)::value;
    const int nb = n0 + 128 * wn + hd * D;   // first column of the head (wave-uniform)
    if (nb >= a.N) {
    } else if (nb < a.C_kv) {
      // ---- q, k or v head: conv, SiLU, (queries and keys) L2 norm
      const bool is_q = nb < a.C_q;
      const bool is_k = nb < a.C_k;   // q or k: normalised
      if (any_tail) {
        // the raw projection of the segment's last w-1 rows is the conv state
        static_for<JB>([&](auto jj_c) {
          constexpr int j = hd * JB + decltype(jj_c)::value;
          const float sc = bf16_bits_to_f32(sc_raw[j]);
          const bool pad = rect_k && 32 * j >= a.k_real;
          const int ch = real_col<RECT, D>(a, ncol + 32 * j);
#pragma unroll
          for (int u = 0; u < 32; ++u) {
            if ((tailm >> u) & 1u) {
              const RowInfo r = a.info[t0 + u];
              if (r.slot >= 0 && !pad)
                store_elem(a.tail, ((int64_t)r.slot * a.c_tail + a.tail_kv_off + ch) * w1 + (w1 - r.rem),
                           XU(j, u) * sc, tail_bf16);
            }
          }
        });
      }
      // Rows in descending order, so each x is overwritten only after the
      // three rows after it have read it; one row of the head's blocks per
      // group (the scheduler would otherwise hoist every row's exp and keep
      // all conv results live at once).
      float ss[32];
      auto conv_row = [&](int u, auto mask_tag) {
        constexpr bool MASK = decltype(mask_tag)::value;
        ss[u] = 0.f;
        static_for<JB>([&](auto jj_c) {
          constexpr int j = hd * JB + decltype(jj_c)::value;
          const float x1 = u >= 1 ? XU(j, u - 1) : xp[2][j];
          const float x2 = u >= 2 ? XU(j, u - 2) : xp[u + 1][j];
          const float x3 = u >= 3 ? XU(j, u - 3) : xp[u][j];
          float z = tp[j][0] * XU(j, u);
          z = fmaf(tp[j][1], MASK && !((m1 >> u) & 1u) ? 0.f : x1, z);
          z = fmaf(tp[j][2], MASK && !((m2 >> u) & 1u) ? 0.f : x2, z);
          z = fmaf(tp[j][3], MASK && !((m3 >> u) & 1u) ? 0.f : x3, z);
          float y = z * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(z));   // -SiLU / ln2
          asm volatile("" : "+v"(y));   // materialise y here (not z and 1/(1+2^z) until the stores)
          XU(j, u) = y;
          ss[u] = fmaf(y, y, ss[u]);
        });
      };
#pragma unroll
      for (int u = 31; u >= 0; --u) {
        if ((cmask >> u) & 1u) conv_row(u, std::true_type{});
        else conv_row(u, std::false_type{});
        __builtin_amdgcn_sched_barrier(0);
      }
      if (is_k) {
        // sum of squares of each row over the head's D columns: over the
        // lane's blocks above, then across the 32 lanes of the half-wave
        // (reduce-scatter: lane lc ends with the total of row bitrev5(lc))
        bfly_step<32, 0, 0xB1>(ss, lc);    // quad_perm 1,0,3,2: lane ^ 1
        bfly_step<16, 1, 0x4E>(ss, lc);    // quad_perm 2,3,0,1: lane ^ 2
        bfly_step<8, 2, 0x124>(ss, lc);    // row_ror 4: bit 2 flipped
        bfly_step<4, 3, 0x128>(ss, lc);    // row_ror 8: lane ^ 8
        bfly_step<2, 4, -1>(ss, lc);       // swizzle: lane ^ 16
        const int tau = (int)(__builtin_bitreverse32((uint32_t)lc) >> 27);
        INV[((wid * 2 + hf) * NH + hd) * 32 + tau] =
            (is_q ? -kLn2 * a.q_scale : -kLn2) * __builtin_amdgcn_rsqf(kLn2 * kLn2 * ss[0] + a.eps);
        __builtin_amdgcn_s_waitcnt(0xc07f);
      }
      // scale (1/|k| for keys), round to bf16, store two rows per pack
      const int hh = is_q ? nb / D : (is_k ? (nb - a.C_q) / D : (nb - a.C_k) / D);
      uint16_t* dst = static_cast<uint16_t*>(is_q ? a.Qbuf : (is_k ? a.Kbuf : a.Vbuf)) + ((int64_t)hh * T + t0) * D + lc;
      // RECT values: value head h (v_head = 2 k_real columns) is stored as
      // two halves h 2 + e of k_real columns, each padded to D like a key
      // head ([2 H_v][T][D]).  Block jj of these 128 columns is columns
      // col .. col + 31 of half vh; the block ending a half also writes the
      // half's pad columns (zeros).
      uint16_t* vdst[JB];
      bool vpad[JB];
      if constexpr (RECT) {
        if (!is_k) {
#pragma unroll
          for (int jj = 0; jj < JB; ++jj) {
            const int c = nb - a.C_k + 32 * jj, h = c / a.v_head, j0 = c - h * a.v_head;
            const int e = j0 / a.k_real, col = j0 - e * a.k_real;
            vdst[jj] = static_cast<uint16_t*>(a.Vbuf) + ((int64_t)(2 * h + e) * T + t0) * D + col + lc;
            vpad[jj] = col + 32 == a.k_real;
          }
        }
      }
      const lfloat* ivp = INV + ((wid * 2 + hf) * NH + hd) * 32;
      // SIMPLE: every lane outputs rows 3..31, so only rows 0-2 need a
      // per-lane predicate
      auto out_pass = [&](auto simple_tag) {
        constexpr bool SIMPLE = decltype(simple_tag)::value;
        auto st = [&](uint16_t* p, uint16_t v, int u) {
          if (SIMPLE && u >= HALO) *p = v;
          else row_store(p, v, u);
        };
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          nf32x4 iv = nf32x4{-kLn2, -kLn2, -kLn2, -kLn2};
          if (is_k) iv = *reinterpret_cast<const __attribute__((address_space(3))) nf32x4*>(ivp + 4 * q);
          static_for<JB>([&](auto jj_c) {
            constexpr int jj = decltype(jj_c)::value, j = hd * JB + jj;
#pragma unroll
            for (int v = 0; v < 4; v += 2) {
              const int u = 4 * q + v;
              const uint32_t p = pack_bf16x2(XU(j, u) * iv[v], XU(j, u + 1) * iv[v + 1]);
              if (RECT && !is_k) {
                st(vdst[jj] + (int64_t)u * D, (uint16_t)(p & 0xffffu), u);
                st(vdst[jj] + (int64_t)(u + 1) * D, (uint16_t)(p >> 16), u + 1);
                if (vpad[jj]) {
                  st(vdst[jj] + (int64_t)u * D + 32, (uint16_t)0, u);
                  st(vdst[jj] + (int64_t)(u + 1) * D + 32, (uint16_t)0, u + 1);
                }
              } else {
                st(dst + (int64_t)u * D + 32 * jj, (uint16_t)(p & 0xffffu), u);
                st(dst + (int64_t)(u + 1) * D + 32 * jj, (uint16_t)(p >> 16), u + 1);
              }
            }
          });
        }
      };
      if ((ofull | 7u) == ~0u) out_pass(std::true_type{});
      else out_pass(std::false_type{});
    } else if (nb < a.C_z) {
      // ---- z head (output gate): the raw projection, bf16, head-major
      uint16_t* dst = static_cast<uint16_t*>(a.Zbuf) + ((int64_t)((nb - a.C_kv) / D) * T + t0) * D + lc;
#pragma unroll
      for (int u = 0; u < 32; u += 2) {
        static_for<JB>([&](auto jj_c) {
          constexpr int jj = decltype(jj_c)::value, j = hd * JB + jj;
          const float sc = bf16_bits_to_f32(sc_raw[j]);
          const uint32_t p = pack_bf16x2(XU(j, u) * sc, XU(j, u + 1) * sc);
          row_store(dst + (int64_t)u * D + 32 * jj, (uint16_t)(p & 0xffffu), u);
          row_store(dst + (int64_t)(u + 1) * D + 32 * jj, (uint16_t)(p >> 16), u + 1);
        });
      }
    } else {
      // ---- gate columns: G = log2 alpha from a, beta from b (no conv).  G
      // and beta are head-major ([H_v][T]), so a lane's 32 rows of one
      // column are 32 scattered rows for the wave: each 32-column block is
      // transposed through the wave's LDS area and stored 64 rows of one
      // head at a time.  Every row of the tile from HALO on that lies
      // before T is an output (gates do not depend on the segments).
      lfloat* tw = (lfloat*)smem_raw + wid * 32 * GATE_PITCH;
      const int64_t trow = row0 + wm * 64 + lane;   // the row this lane stores
      const bool st_ok = wm * 64 + lane >= HALO && trow < T;
      static_for<JB>([&](auto jj_c) {
        constexpr int j = hd * JB + decltype(jj_c)::value;
        const int nb_j = n0 + 128 * wn + 32 * j;   // first column of the block (wave-uniform)
        if (nb_j < a.N) {
          const int n = ncol + 32 * j;
          const float sc = bf16_bits_to_f32(sc_raw[j]);
          const bool is_a = n < a.C_z + a.H_v;
          const int hv = is_a ? n - a.C_z : n - a.C_z - a.H_v;
          float al = 0.f, db = 0.f;
          if (n < a.N && is_a) {
            al = -__expf(a.a_log[hv]) * kLog2e;
            db = a.dt_bias[hv];
          }
          lfloat* col = tw + lc * GATE_PITCH + 32 * hf;
#pragma unroll
          for (int u = 0; u < 32; u += 4) {
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float x = XU(j, u + e) * sc;
              v[e] = is_a ? al * softplus(x + db) : fast_sigmoid(x);
            }
            st_f4(col + u, v[0], v[1], v[2], v[3]);
          }
          // LDS operations of one wave complete in order: the reads below
          // see every lane's writes
          const int nc = a.N - nb_j < 32 ? a.N - nb_j : 32;
          for (int c = 0; c < nc; ++c) {
            const int nn = nb_j + c;
            const bool ca = nn < a.C_z + a.H_v;
            float* dst = ca ? a.Gbuf + (int64_t)(nn - a.C_z) * T : a.Bbuf + (int64_t)(nn - a.C_z - a.H_v) * T;
            const float v = tw[c * GATE_PITCH + lane];
            if (st_ok) dst[trow] = v;
          }
        }
      });
    }
  });
#undef XU
}

template <typename TB, int D, bool RECT = false>
hipError_t run(const ProjConvBatch& b, hipStream_t s) {
  const ProjConvArgs& a = b.layer[0];
  if (a.K % BK) return hipErrorInvalidValue;
  const int tm = (int)((a.T + SM - 1) / SM), tn = (a.N + BN - 1) / BN;
  const int blocks = b.n_layers * tm * tn + b.tq_off[b.n_layers];
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL((proj_conv_kernel<TB, D, RECT>), dim3(blocks), dim3(THREADS), 0, s, b, tm, tn);
  return hipGetLastError();
}

template <typename TB>
hipError_t by_head(int d, const ProjConvBatch& a, hipStream_t s) {
  if (a.layer[0].k_real > 0) {
    // rectangular heads: key heads padded to 128 columns, no q or z columns
    for (int l = 0; l < a.n_layers; ++l) {
      const ProjConvArgs& x = a.layer[l];
      if (x.k_real != a.layer[0].k_real || x.v_head != a.layer[0].v_head || x.k_real % 32 || x.k_real >= 128 ||
          x.k_real + 32 != 128 || x.v_head != 2 * x.k_real || x.C_q != 0 || x.C_z != x.C_kv || x.C_k % 128 ||
          (x.C_kv - x.C_k) % 128)
        return hipErrorInvalidValue;
    }
    return d == 128 ? run<TB, 128, true>(a, s) : hipErrorInvalidValue;
  }
  switch (d) {
    case 32: return run<TB, 32>(a, s);
    case 64: return run<TB, 64>(a, s);
    case 128: return run<TB, 128>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_proj_conv(int weight_dtype, int d_head, const ProjConvBatch& b, hipStream_t s) {
  if (b.n_layers < 1 || b.n_layers > kProjBatch) return hipErrorInvalidValue;
  for (int l = 1; l < b.n_layers; ++l)
    if (b.layer[l].T != b.layer[0].T || b.layer[l].K != b.layer[0].K || b.layer[l].N != b.layer[0].N)
      return hipErrorInvalidValue;
  if (weight_dtype == SR_BF16) return by_head<bf16_t>(d_head, b, s);
  if (weight_dtype == SR_FP8_E4M3) return by_head<fp8_t>(d_head, b, s);
  return hipErrorInvalidValue;
}

hipError_t launch_proj_conv(int weight_dtype, int d_head, const ProjConvArgs& a, hipStream_t s) {
  ProjConvBatch b{};
  b.layer[0] = a;
  b.n_layers = 1;
  b.tq_off[1] = a.tq_blocks;
  return launch_proj_conv(weight_dtype, d_head, b, s);
}

}  // namespace sr
