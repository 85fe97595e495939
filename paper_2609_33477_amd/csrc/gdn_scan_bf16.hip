// Chunked Gated DeltaNet state accumulation, bf16 operands (gfx950).
//
// Same recurrence as the fp32 kernel (gdn_scan.hip).  Rows go 32 at a time
// (a sub-chunk); a sub-chunk that starts from state M0 (= S^T), with G the
// sub-chunk prefix of log2 alpha, does
//   A_ij  = beta_i 2^{G_i - G_j} k_i.k_j  (i > j)        T = (I + A)^{-1}  (32x32)
//   U     = T diag(beta) V,    W = T diag(beta 2^G) K
//   Delta = U - W M0
//   M_32  = 2^{G_31} M0 + K^T diag(2^{G_31 - G}) Delta
// Only the last two lines touch the state.  The workgroup runs a pipeline
// with one barrier per sub-chunk step:
//   4 prep waves: wave p builds everything but the state lines for the
//     sub-chunk pairs (m, m+1), m = 2p (mod 8), over the 8 steps m-9 .. m-2,
//     lanes 0-31 serving sub-chunk m and lanes 32-63 sub-chunk m+1 wherever
//     the work is one lane per row or column: K rows for the Gram blocks
//     straight from global memory (issued two steps ahead); log2-alpha
//     prefix and Gram blocks on MFMA (step m-8); A (m-7); T = (I + A)^{-1}
//     by a 32-step forward substitution in fp32, lane = column of T, spread
//     over steps m-6 .. m-4; Tu = T diag(beta) in two bf16 parts and
//     Tw = T diag(beta 2^G) (m-3); then W^T = K^T Tw^T, which leaves W
//     row-major (m-2 for sub-chunk m, m-1 for m+1);
//   d/32 state waves, wave s owning state columns [32s, 32s+32) as 2 d/16
//     16x16 fp32 accumulator tiles for the whole unit: at step n they
//     run the state lines of sub-chunk n from registers (in phases that
//     pair MFMA groups with the VALU work they do not wait on), then read
//     the operands of sub-chunk n+1, so the reads' latency overlaps the
//     MFMAs and the barrier.
// K(n+5) and V(n+4) go global -> LDS by DMA, requested at step n by the prep
// wave whose phase there is Gram or A (the two lightest) and waited for two
// steps later, so the state waves issue nothing but LDS reads and MFMAs.
// Rings (sub-chunk slots): K 5, V 4, W 2, Tu 4, gate vectors 16.
//
// The grid is one workgroup per CU.  A workgroup runs its units (segment,
// layer, value head) back to back as one stream of sub-chunks: the pipeline
// does not drain between units, so a unit of a few sub-chunks does not pay
// the 9 steps of pipeline fill.  Each reference to sub-chunk j of the stream
// goes through a cursor that caches its unit's rows and planes in scalar
// registers; the state waves start a unit's state at its first sub-chunk and
// store it after its last.
//
// Every product is v_mfma_f32_16x16x32_bf16.  A 32-wide reduction over
// sub-chunk rows uses the k-slot order {4g..4g+3, 16+4g..16+4g+3} for lane
// group g, which is the row order of two stacked 16x16 accumulator tiles,
// so Delta and the state feed later products straight from accumulator
// registers; operands whose reduction index runs down the rows of an LDS
// matrix are read with ds_read_b64_tr_b16, which hands lane i of each
// 16-lane group rows kbase..kbase+3 of column n0 + i when lane j of the group
// addresses row kbase + j/4, columns n0 + 4 (j%4) .. +3.
//
// LDS (d = 128): K and V rings 72 KB, W ring 18 KB, Tu ring 24 KB, gate
// vectors 4 KB, per prep wave A^T of a pair (reused for Tw^T) and gate
// scratch 38 KB: ~159 KB, one workgroup (8 waves) per CU.  K and V rows are
// unpadded and XOR-swizzled (kv_off) so the DMA writes whole 1 KB blocks;
// W rows hold their columns in the state's k order (32q + 4g .. + 3, then
// 32q + 16 + 4g .. + 3, at 32q + 8g) so each fragment is one 16-byte read,
// with the row pitch 8 mod 64 dwords measured conflict free for those.
//
// Rectangular heads (SPLIT, d = 128): OLMo-Hybrid's 192-wide value heads
// arrive as two 96-column halves and its 96-wide keys as 128-column rows,
// all padded with zeros.  Each half runs as a unit of its own with the head's
// G, beta and key head; zero key columns leave Gram, T and W those of the
// real keys, zero value columns stay zero in the state, and the unit reads
// and writes only its 96 x 96 block of the head's [96][192] state.
#include "sr_device.hpp"

#include <cstddef>

namespace sr {
namespace {

constexpr int kC = 64;       // rows staged per step
constexpr int kScanUnits = 64;   // units one workgroup runs at most (one wave's lanes: the prefix is a wave scan)
constexpr int kS = 32;       // sub-chunk rows
constexpr int kAP = 36;      // fp32 pitch of a sub-chunk's A (rows read as float4)
constexpr int kTP = 48;      // bf16 pitch of the T^T blocks (transposed reads)

typedef short v4i16 __attribute__((ext_vector_type(4)));

// LDS is addressed through address-space-3 pointers with 32-bit offsets so
// that per-read constants fold into the instructions' offset field.
#define SR_LDS __attribute__((address_space(3)))
typedef SR_LDS char lchar;
typedef unsigned int nu32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int nu32x2 __attribute__((ext_vector_type(2)));
typedef float nf32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 lds_ld16(const lchar* p) {
  return __builtin_bit_cast(uint4, *reinterpret_cast<const SR_LDS nu32x4*>(p));
}
__device__ __forceinline__ uint2 lds_ld8(const lchar* p) {
  return __builtin_bit_cast(uint2, *reinterpret_cast<const SR_LDS nu32x2*>(p));
}
__device__ __forceinline__ float4 lds_ldf4(const lchar* p) {
  const nf32x4 v = *reinterpret_cast<const SR_LDS nf32x4*>(p);
  return make_float4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void lds_st16(lchar* p, const uint4& v) {
  *reinterpret_cast<SR_LDS nu32x4*>(p) = __builtin_bit_cast(nu32x4, v);
}
__device__ __forceinline__ void lds_stf4(lchar* p, const float* v) {
  *reinterpret_cast<SR_LDS nf32x4*>(p) = nf32x4{v[0], v[1], v[2], v[3]};
}
__device__ __forceinline__ void lds_st8(lchar* p, const uint2& v) {
  *reinterpret_cast<SR_LDS nu32x2*>(p) = __builtin_bit_cast(nu32x2, v);
}

__device__ __forceinline__ bf16x8 join(uint2 lo, uint2 hi, bool negate) {
  uint4 u = make_uint4(lo.x, lo.y, hi.x, hi.y);
  if (negate) { u.x ^= 0x80008000u; u.y ^= 0x80008000u; u.z ^= 0x80008000u; u.w ^= 0x80008000u; }
  return as_bf16x8(u);
}

__device__ __forceinline__ v4i16 as_v4(uint2 u) { return __builtin_bit_cast(v4i16, u); }

// Two 16x16 accumulator tiles (rows 4g..4g+3 of each) as one 16x16x32 operand.
__device__ __forceinline__ bf16x8 acc_pair(const f32x4& x, const f32x4& y) {
  return as_bf16x8(make_uint4(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(y[0], y[1]),
                              pack_bf16x2(y[2], y[3])));
}

__device__ __forceinline__ f32x4 mma_k32(const f32x4& c, const bf16x8& a, const bf16x8& b) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma_k16(const f32x4& c, const v4i16& a, const v4i16& b) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// value of lane - N inside the lane's 16-lane row (0 for the first N lanes)
template <int N>
__device__ __forceinline__ float dpp_row_shr(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x110 + N, 0xf, 0xf, false));
}
// value at lane 15 of 16-lane row `row` (0..3); every lane of the wave calls it
__device__ __forceinline__ float row_last(float x, int row) {
  const int v = __builtin_bit_cast(int, x);
  const int r0 = __builtin_amdgcn_readlane(v, 15), r1 = __builtin_amdgcn_readlane(v, 31);
  const int r2 = __builtin_amdgcn_readlane(v, 47), r3 = __builtin_amdgcn_readlane(v, 63);
  return __builtin_bit_cast(float, row == 0 ? r0 : row == 1 ? r1 : row == 2 ? r2 : r3);
}

template <int D>
struct Cfg {
  static constexpr int NSW = D / 32;                  // state waves; wave s owns columns [32s, 32s+32)
  static constexpr int NP = 4;                        // prep waves
  static constexpr int THREADS = 64 * (NSW + NP);
  static constexpr int NT = D / 16;                   // 16-row tiles along d
  // K and V sub-chunks: unpadded rows of 2D bytes, 32-byte chunk pairs
  // XOR-swizzled by row (see kv_off), staged by global -> LDS DMA
  static constexpr int RPL = 128 / D;                 // rows per 256-byte bank line
  static constexpr int NCP = D / 16;                  // 32-byte chunk pairs per row
  static constexpr int DMA_ROWS = 512 / D;            // rows per 1 KB DMA block
  static constexpr int DMA_BLK = kS * 2 * D / 1024;         // 1 KB DMA blocks of one K or V sub-chunk
  static constexpr int WP = D + 16;                   // W row pitch (bf16): 16-byte row reads
  static constexpr int NK = 5;                        // K ring: K(n) DMA issued at step n-5
  static constexpr int NV = 4;                        // V ring: V(n) DMA issued at step n-4
  static constexpr int NTU = 4;                       // Tu ring: a pair is packed two steps ahead
  static constexpr int NVEC = 16;                     // gate-vector ring: written nine steps ahead
  static constexpr int SZ_KV = kS * D * 2;            // one sub-chunk of K or V
  static constexpr int SZ_W = kS * WP * 2;
  static constexpr int SZ_TT = kS * kTP * 2;          // one T^T block (bf16)
  static constexpr int SZ_A = kS * kAP * 4;           // A^T of one sub-chunk (fp32)
  static constexpr int SZ_VEC = 2 * kS * 4;           // eD[32] | 2^{G_31}
  static constexpr int SZ_GB = 2 * kS * 4;            // G prefix[32] | beta[32] of one sub-chunk
  // private area of a prep wave: A^T of its two sub-chunks (later Tw^T of
  // both), then their G prefix and beta
  static constexpr int SZ_PRIV = 2 * SZ_A + 2 * SZ_GB;
  static constexpr int OFF_K = 0;
  static constexpr int OFF_V = OFF_K + NK * SZ_KV;
  static constexpr int OFF_W = OFF_V + NV * SZ_KV;
  static constexpr int OFF_TU = OFF_W + 2 * SZ_W;     // slot: Tu_hi^T | Tu_lo^T
  static constexpr int OFF_VEC = OFF_TU + NTU * 2 * SZ_TT;
  static constexpr int OFF_PRIV = OFF_VEC + NVEC * SZ_VEC;
  static constexpr int LDS = OFF_PRIV + NP * SZ_PRIV;
  static constexpr int QG = D / 32;                   // 32-wide d blocks (Gram k-steps)
  static_assert(DMA_BLK * 1024 == kS * 2 * D, "staging split");
  static_assert(NT % 2 == 0, "state tiles pair up along d");
  static_assert(2 * SZ_TT <= 2 * SZ_A, "Tw^T of both sub-chunks reuses the A^T area");
  static_assert(LDS <= 160 * 1024, "LDS");
};

// Byte offset of the 8 bytes at row r, columns 16 cb + 4 h .. + 3 (h = 0..3)
// of a K or V sub-chunk.  Rows are unpadded (2D bytes) and the 32-byte
// column pair cb of row r is stored at pair cb ^ ((r / RPL) mod NCP): the 8
// consecutive rows that the 16-lane groups of a transposed read cover then
// fall on 8 distinct groups of 8 banks, as with a row pitch of 8 mod 64 dwords.
template <int D>
__device__ __forceinline__ int kv_off(int r, int cb, int h) {
  constexpr int RPL = Cfg<D>::RPL, NCP = Cfg<D>::NCP;
  return r * 2 * D + 32 * (cb ^ ((r / RPL) % NCP)) + 8 * h;
}

// SPLIT: value heads run as several units (the v_split fields of ScanArgs);
// the square-head kernels are built without it.
template <int D, bool SPLIT>
__global__ __launch_bounds__(64 * (D / 32 + 4), 1) void gdn_scan_bf16_kernel(ScanArgs a) {
  if (a.err && *a.err) return;   // the call's table check failed: write nothing
  using CF = Cfg<D>;
  constexpr int NSW = CF::NSW, NP = CF::NP, NT = CF::NT, WP = CF::WP, NK = CF::NK, NV = CF::NV, QG = CF::QG;
  __shared__ __attribute__((aligned(16))) char smem[CF::LDS];
  __shared__ int seg_of[kSortMax];                 // rank -> segment, longest first
  __shared__ int seg_len[kSortMax];                // segment lengths (-1: sentinel)
  // the block's units, in the order it runs them, and where each one's
  // sub-chunks start in the block's stream (u_p[k] .. u_p[k+1] - 1)
  __shared__ int u_s0[kScanUnits], u_s1[kScanUnits], u_lh[kScanUnits], u_slot[kScanUnits];
  __shared__ int u_p[kScanUnits + 1];

  lchar* L = (lchar*)smem;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, li = lane & 15;
  // per-lane byte offsets; everything else is a compile-time immediate
  const int w_row = (li * WP + 8 * g) * 2;                            // W rows: 8-byte writes, 16-byte reads
  const int tr_row = 4 * g + (li >> 2);                              // transposed reads of K / V: row, 8-byte piece
  const int tr_h = li & 3;
  const int tr_t = ((li >> 2) * kTP + 4 * (li & 3) + 4 * g * kTP) * 2; // transposed reads of T^T, rows 4g + ..

  // ---- the block's units.  Unit (rank, layer, value head), ranks longest
  // first, are dealt in rounds of G (the grid): round k gives block b unit
  // kG + pi(b) (k even) or kG + G - 1 - pi(b) (k odd), a snake, so a block
  // with a long unit in one round takes a short one in the next.  Blocks are
  // dealt to the 8 XCDs round-robin; pi pairs blocks r and r + 8 of each 16
  // (same XCD, dispatched together) on consecutive units, value heads 2i and
  // 2i + 1, which share a key head when H_v = 2 H_k, so its K rows are
  // fetched into one L2.
  const int units = a.n_seg * a.n_layers * a.H_v;
  const int G = gridDim.x, bid = blockIdx.x;
  const int pi = (G & 15) == 0 ? (bid & ~15) + 2 * (bid & 7) + ((bid >> 3) & 1) : bid;
  if (a.n_seg <= kSortMax) {
    for (int sg = tid; sg < a.n_seg; sg += CF::THREADS) {
      const int sl = a.slot_ids ? a.slot_ids[sg] : sg;
      seg_len[sg] = sl < 0 ? -1 : a.cu[sg + 1] - a.cu[sg];
    }
    __syncthreads();
    for (int sg = tid; sg < a.n_seg; sg += CF::THREADS) {
      const int ls = seg_len[sg];
      int r = 0;
      for (int s2 = 0; s2 < a.n_seg; ++s2) {
        const int l2 = seg_len[s2];
        r += (l2 > ls) || (l2 == ls && s2 < sg);
      }
      seg_of[r] = sg;
    }
  }
  __syncthreads();
  const int n_rounds = (units + G - 1) / G;   // units this block may hold (<= kScanUnits)
  if (tid < kScanUnits) {
    const int k = tid;
    const int uk = k * G + ((k & 1) ? G - 1 - pi : pi);
    int nsc_k = 0, s0k = 0, s1k = 0, lh = 0, sl = -1;
    if (uk < units) {
      const int head = uk % a.H_v, layer = (uk / a.H_v) % a.n_layers, rank = uk / (a.H_v * a.n_layers);
      const int sg = a.n_seg <= kSortMax ? seg_of[rank] : rank;
      sl = a.slot_ids ? a.slot_ids[sg] : sg;
      s0k = a.cu[sg];
      s1k = a.cu[sg + 1];
      lh = layer * a.H_v + head;
      if (sl >= 0) nsc_k = (s1k - s0k + kS - 1) / kS;
    }
    u_s0[k] = s0k;
    u_s1[k] = s1k;
    u_lh[k] = lh;
    u_slot[k] = sl;
    u_p[k + 1] = nsc_k;   // prefix summed below
  }
  __syncthreads();
  if (tid < 64) {   // inclusive prefix over the 64 entries, one per lane of wave 0
    int v = u_p[tid + 1];
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int y = __shfl_up(v, off);
      if (tid >= off) v += y;
    }
    u_p[tid + 1] = v;
    if (tid == 0) u_p[0] = 0;
  }
  __syncthreads();
  // the tables are the same for every lane: their reads go to scalar registers
  auto uni = [](int v) { return __builtin_amdgcn_readfirstlane(v); };
  const int NSC = uni(u_p[kScanUnits]);   // sub-chunks of the block's stream
  // a unit's state pointers (layer l of this launch) from the kernel-argument
  // segment at a uniform offset (ScanArgs is the only argument, at offset 0)
  const char* kargs = (const char*)__builtin_amdgcn_kernarg_segment_ptr();
  auto st_in_of = [&](int layer) {
    return *reinterpret_cast<const float* const*>(kargs + offsetof(ScanArgs, state_in) + sizeof(void*) * layer);
  };
  auto st_out_of = [&](int layer) {
    return *reinterpret_cast<float* const*>(kargs + offsetof(ScanArgs, state_out) + sizeof(void*) * layer);
  };
  // Where a unit's state lives: value heads of v_split units each, the
  // unit's rows < st_rows and columns < st_cols at [row][col] of pitch
  // st_pitch (D, D, D and one unit per head for square heads)
  const int vsp = SPLIT ? a.v_split : 1;
  const int srows = SPLIT ? a.st_rows : D, scols = SPLIT ? a.st_cols : D;
  const int spitch = SPLIT ? a.st_pitch : D;
  auto state_base = [&](int slot, int head) {
    return ((size_t)slot * (a.H_v / vsp) + head / vsp) * srows * spitch + (size_t)(head % vsp) * scols;
  };
  // live units without rows: their state is the initial one
  for (int k = 0; k < n_rounds; ++k) {
    if (u_slot[k] < 0 || u_s1[k] != u_s0[k]) continue;
    const int layer = u_lh[k] / a.H_v, head = u_lh[k] % a.H_v;
    const float* si = st_in_of(layer);
    const size_t ib = state_base(u_slot[k], head);
    float* so = st_out_of(layer) + ib;
    for (int i = tid; i < srows * scols; i += CF::THREADS) {
      const size_t o = (size_t)(i / scols) * spitch + i % scols;
      so[o] = si ? si[ib + o] : 0.f;
    }
  }
  if (NSC == 0) return;

  // Sub-chunk j of the stream: its unit (a cursor that only moves forward,
  // with the unit's stream range, rows and planes cached in scalar
  // registers, so the table is read only when the cursor crosses into the
  // next unit; j past the stream stays in the last unit with sub-chunks,
  // past its rows), first row c0, segment end s1 and the K, V, G, beta planes.
  struct Cursor {
    int k, beg, end;         // unit, its sub-chunks [beg, end) of the stream
    int64_t s0, s1;          // its rows
    const char* kp;
    const char* vp;
    const float* gp;
    const float* bp;
  };
  auto cursor_at = [&](Cursor& c, int k) {
    c.k = k;
    c.beg = uni(u_p[k]);
    c.end = uni(u_p[k + 1]);
    c.s0 = uni(u_s0[k]);
    c.s1 = uni(u_s1[k]);
    const int lh = uni(u_lh[k]);
    const int layer = lh / a.H_v, head = lh % a.H_v;
    const int hk = (head * a.H_k) / a.H_v;
    c.kp = static_cast<const char*>(a.Kbuf) + (layer * a.k_layer_stride + (int64_t)hk * a.T * D) * 2;
    c.vp = static_cast<const char*>(a.Vbuf) + (layer * a.v_layer_stride + (int64_t)head * a.T * D) * 2;
    c.gp = a.Gbuf + layer * a.g_layer_stride + (int64_t)(head / vsp) * a.T;
    c.bp = a.Bbuf + layer * a.g_layer_stride + (int64_t)(head / vsp) * a.T;
  };
  auto cursor_new = [&]() {
    Cursor c;
    int k = 0;
    while (k + 1 < kScanUnits && uni(u_p[k + 1]) == 0) ++k;   // the first unit with sub-chunks
    cursor_at(c, k);
    return c;
  };
  struct Sub {
    const char* kp;
    const char* vp;
    const float* gp;
    const float* bp;
    int64_t c0, s1;
  };
  auto sub = [&](int j, Cursor& c) {
    if (j >= c.end && c.end < NSC) {
      int k = c.k + 1;
      while (k + 1 < kScanUnits && uni(u_p[k + 1]) <= j && uni(u_p[k + 1]) < NSC) ++k;
      cursor_at(c, k);
    }
    Sub r;
    r.kp = c.kp;
    r.vp = c.vp;
    r.gp = c.gp;
    r.bp = c.bp;
    r.c0 = c.s0 + (int64_t)(j - c.beg) * kS;
    r.s1 = c.s1;
    return r;
  };

  auto kbuf = [&](int m) { return L + CF::OFF_K + (m % NK) * CF::SZ_KV; };
  auto vbuf = [&](int m) { return L + CF::OFF_V + (m & (NV - 1)) * CF::SZ_KV; };
  auto wbuf = [&](int m) { return L + CF::OFF_W + (m & 1) * CF::SZ_W; };
  auto tubuf = [&](int m) { return L + CF::OFF_TU + (m & (CF::NTU - 1)) * 2 * CF::SZ_TT; };   // Tu_hi^T, then Tu_lo^T
  auto vecbuf = [&](int m) { return (SR_LDS float*)(L + CF::OFF_VEC + (m & (CF::NVEC - 1)) * CF::SZ_VEC); };

  // A 32-wide reduction operand from a transposed-read matrix: rows
  // kbase + {4g..4g+3} and kbase + 16 + {4g..4g+3} of the lane's column.
  auto tr_pair = [&](const lchar* p, int pitch_bytes, bool negate) {
    return join(lds_tr4(p), lds_tr4(p + 16 * pitch_bytes), negate);
  };
  // the same for column block cb (16 columns) of a K or V sub-chunk
  auto tr_kv = [&](const lchar* base, int cb) { return tr_pair(base + kv_off<D>(tr_row, cb, tr_h), 2 * D, false); };

  if (wid < NP) {
    // ================================================================ prep
    // Wave p prepares the sub-chunk pairs (m, m + 1), m = 2p (mod 8), each
    // over the eight steps m-9 .. m-2 (phase s at step m-9+s) plus W(m+1)
    // at step m-1.  Lanes 0-31 work on sub-chunk m, lanes 32-63 on m + 1 where
    // the work is one lane per row or column (prefix, solve, packing).
    const int p = wid;
    lchar* priv = L + CF::OFF_PRIV + p * CF::SZ_PRIV;
    const int hc = lane >> 5;                            // sub-chunk of the pair this lane serves
    const int col = lane & 31;                           // its row (gates) / column of T (solve)
    SR_LDS float* gsc_l = (SR_LDS float*)(priv + 2 * CF::SZ_A + hc * CF::SZ_GB);   // G prefix | beta
    const SR_LDS float* At_l = (const SR_LDS float*)(priv + hc * CF::SZ_A);         // this lane's A^T

    bf16x8 kf[2][QG][2];   // Gram operands of the pair: [sub-chunk][d block][row half]
    float gv = 0.f, bv = 0.f;
    f32x4 gr[2][3];        // Gram tiles (0,0), (1,0), (1,1) of each sub-chunk
    float x[kS];           // column `col` of T, carried over the solve phases

    // DMA staging of K and V, global -> LDS: at step n the prep wave in its
    // Gram or A phase (the two lightest) requests K(n + 5) and V(n + 4), all
    // DMA_BLK 1 KB blocks of each, and waits for them at the end of step
    // n + 2, before the barrier that publishes them (K(j) is read from step
    // j - 2 on, V(j) at step j - 1): a DMA has the rest of its step and two
    // more to land, which covers its latency under load (one step did not:
    // the A-phase requests then stalled the next phase by ~2K cycles).
    // Lane l carries the 16 bytes at byte 16 l of a block: dma_off is their
    // byte offset from the sub-chunk's first row in the swizzled layout.  Rows past the segment end are read from
    // its last row: their beta and log decay are 0, so T has unit rows and
    // zero columns there and any finite values are multiplied by exact zeros.
    uint32_t dma_off[CF::DMA_BLK];
#pragma unroll
    for (int i = 0; i < CF::DMA_BLK; ++i) {
      const int byte = i * 1024 + 16 * lane;
      const int r = byte / (2 * D), pos = byte % (2 * D);
      const int cbp = (pos / 32) ^ ((r / CF::RPL) % CF::NCP);
      dma_off[i] = (uint32_t)((r * D + 16 * cbp + 8 * ((pos / 16) & 1)) * 2);
    }
    auto stage = [&](const char* plane, int64_t c0, int64_t s1, lchar* buf) {
      const char* base = plane + c0 * D * 2;
      const uint32_t lds0 = (uint32_t)(uintptr_t)buf;
      if (c0 + kS <= s1) {
#pragma unroll
        for (int i = 0; i < CF::DMA_BLK; ++i) dma16_s(base, dma_off[i], lds0 + i * 1024);
      } else {
        const uint32_t last = (uint32_t)(s1 - 1 - c0);
#pragma unroll
        for (int i = 0; i < CF::DMA_BLK; ++i) {
          const uint32_t r = dma_off[i] / (2 * D), rc = r < last ? r : last;
          dma16_s(base, dma_off[i] - (r - rc) * (2 * D), lds0 + i * 1024);
        }
      }
    };
    // the owner of step n: the wave whose phase there is its Gram (even n)
    // or its A (odd n)
    auto dma_owner = [](int nn) { return ((nn - (nn & 1)) >> 1) & 3; };
    int n = -9;                      // the step; every prep barrier advances it
    int dma_cur = 0, dma_prev = 0, dma_prev2 = 0;   // blocks this wave requested in this / the previous / the step before
    Cursor cur_k = cursor_new(), cur_v = cur_k, cur_l = cur_k;   // of the K and V DMAs and of the Gram loads
    int64_t pc0[2] = {0, 0}, ps1[2] = {0, 0};   // first row and segment end of the pair being loaded
    auto dma_duty = [&](int nn) {
      if (dma_owner(nn) != p) return;
      if (nn + 5 >= 0 && nn + 5 < NSC) {
        const Sub sk = sub(nn + 5, cur_k);
        stage(sk.kp, sk.c0, sk.s1, kbuf(nn + 5));
        dma_cur += CF::DMA_BLK;
      }
      if (nn + 4 >= 0 && nn + 4 < NSC) {
        const Sub sv = sub(nn + 4, cur_v);
        stage(sv.vp, sv.c0, sv.s1, vbuf(nn + 4));
        dma_cur += CF::DMA_BLK;
      }
    };
    // the barrier that ends step nn: the requests of step nn - 2 have
    // landed (those of this step and the previous one may still be in
    // flight; a wave requests on two consecutive steps, then not for six)
    auto pbar = [&](int& nn) {
      if (dma_prev2) {
        const int newer = dma_cur + dma_prev;
        if (newer == 0) wait_vm<0>();
        else if (newer == CF::DMA_BLK) wait_vm<CF::DMA_BLK>();
        else if (newer == 2 * CF::DMA_BLK) wait_vm<2 * CF::DMA_BLK>();
        else if (newer == 3 * CF::DMA_BLK) wait_vm<3 * CF::DMA_BLK>();
        else wait_vm<4 * CF::DMA_BLK>();
      }
      lds_barrier();
      ++nn;
      dma_prev2 = dma_prev;
      dma_prev = dma_cur;
      dma_cur = 0;
    };

    // phase 7 of the previous pair: the pair's K rows straight from global
    // memory as Gram fragments, and this lane's log2 alpha and beta.  Rows
    // past the segment end carry log2 alpha 0 and beta 0, which makes them
    // inert: their K rows are read from the segment's last row (any finite
    // values do, they only meet beta = 0), so every load is unconditional.
    auto issue_loads = [&](int m) {
      const Sub sp[2] = {sub(m, cur_l), sub(m + 1, cur_l)};
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        pc0[c] = sp[c].c0;
        ps1[c] = sp[c].s1;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int64_t t = sp[c].c0 + 16 * h + li;
          const char* rp = sp[c].kp + ((t < sp[c].s1 ? t : sp[c].s1 - 1) * D + 8 * g) * 2;
#pragma unroll
          for (int q = 0; q < QG; ++q) kf[c][q][h] = *reinterpret_cast<const bf16x8*>(rp + 64 * q);
        }
      }
      // raw values of the row (clamped); zeroed past the end in the Gram
      // phase, where they are first used, so nothing here waits for them
      const int64_t t = (hc ? sp[1].c0 : sp[0].c0) + col;
      const int64_t sh = hc ? sp[1].s1 : sp[0].s1;
      const int64_t tc = t < sh ? t : sh - 1;
      gv = (hc ? sp[1].gp : sp[0].gp)[tc];
      bv = (hc ? sp[1].bp : sp[0].bp)[tc];
    };
    // phase 1: prefix of log2 alpha inside each half, gate vectors, Gram
    auto gram = [&](int m) {
      if ((hc ? pc0[1] : pc0[0]) + col >= (hc ? ps1[1] : ps1[0])) {
        gv = 0.f;
        bv = 0.f;
      }
      float gp = gv;
      gp += dpp_row_shr<1>(gp);
      gp += dpp_row_shr<2>(gp);
      gp += dpp_row_shr<4>(gp);
      gp += dpp_row_shr<8>(gp);
      const float g15 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, gp), 15));
      const float g47 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, gp), 47));
      if (col >= 16) gp += hc ? g47 : g15;
      const float g31 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, gp), 31));
      const float g63 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, gp), 63));
      const float glast = hc ? g63 : g31;
      SR_LDS float* vec = vecbuf(m + hc);
      gsc_l[col] = gp;
      gsc_l[kS + col] = bv;
      vec[col] = exp2f(glast - gp);           // 2^{G_31 - G_i}
      if (col == kS - 1) vec[kS] = exp2f(gp); // 2^{G_31}
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        f32x4 g00 = zero4(), g10 = zero4(), g11 = zero4();
#pragma unroll
        for (int q = 0; q < QG; ++q) {
          g00 = mma_k32(g00, kf[c][q][0], kf[c][q][0]);
          g10 = mma_k32(g10, kf[c][q][1], kf[c][q][0]);
          g11 = mma_k32(g11, kf[c][q][1], kf[c][q][1]);
        }
        gr[c][0] = g00;
        gr[c][1] = g10;
        gr[c][2] = g11;
      }
    };
    // phase 2: A_ij = beta_i 2^{G_i - G_j} Gram_ij (i > j), stored
    // transposed, At[j][i] = A_ij: one 16-byte store per 16x16 block
    auto make_a = [&]() {
      // both sub-chunks' gate values first (the compiler cannot move these
      // reads above the A stores, which it cannot tell apart)
      float gj[2][2];
      float4 gi[2][2], bi[2][2];
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const SR_LDS float* gs = (const SR_LDS float*)(priv + 2 * CF::SZ_A + c * CF::SZ_GB);
        gj[c][0] = gs[li];
        gj[c][1] = gs[16 + li];
        gi[c][0] = lds_ldf4((const lchar*)(gs + 4 * g));
        gi[c][1] = lds_ldf4((const lchar*)(gs + 16 + 4 * g));
        bi[c][0] = lds_ldf4((const lchar*)(gs + kS + 4 * g));
        bi[c][1] = lds_ldf4((const lchar*)(gs + kS + 16 + 4 * g));
      }
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        SR_LDS float* At = (SR_LDS float*)(priv + c * CF::SZ_A);
        const float gj0 = gj[c][0], gj1 = gj[c][1];
        const float gi0v[4] = {gi[c][0].x, gi[c][0].y, gi[c][0].z, gi[c][0].w};
        const float gi1v[4] = {gi[c][1].x, gi[c][1].y, gi[c][1].z, gi[c][1].w};
        const float bi0v[4] = {bi[c][0].x, bi[c][0].y, bi[c][0].z, bi[c][0].w};
        const float bi1v[4] = {bi[c][1].x, bi[c][1].y, bi[c][1].z, bi[c][1].w};
        float a00[4], a10[4], a11[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i0 = 4 * g + r, i1 = 16 + 4 * g + r;
          a00[r] = (i0 > li) ? bi0v[r] * exp2f(fminf(gi0v[r] - gj0, 0.f)) * gr[c][0][r] : 0.f;
          a10[r] = bi1v[r] * exp2f(fminf(gi1v[r] - gj0, 0.f)) * gr[c][1][r];
          a11[r] = (i1 > 16 + li) ? bi1v[r] * exp2f(fminf(gi1v[r] - gj1, 0.f)) * gr[c][2][r] : 0.f;
        }
        lds_stf4((lchar*)(At + li * kAP + 4 * g), a00);
        lds_stf4((lchar*)(At + li * kAP + 16 + 4 * g), a10);
        lds_stf4((lchar*)(At + (16 + li) * kAP + 16 + 4 * g), a11);
      }
    };
    // phases 3-5: T = (I + A)^{-1}, lane = column, column-oriented: once
    // x_q = T[q][col] is final it is eliminated from every later row.  Each
    // step needs one column of A (a row of A^T), read two steps ahead, so
    // the pipeline runs on across the phase barriers (the first two columns
    // are read at the end of phase 2).  The empty asm keeps each step's
    // updates in place (later loads may not be hoisted above them, nor the
    // updates sunk below).
    float4 cb[3][kS / 4];
    auto load_col = [&](int q, float4* dst) {
#pragma unroll
      for (int v = (q + 1) / 4; v < kS / 4; ++v) dst[v] = lds_ldf4((const lchar*)(At_l + q * kAP + 4 * v));
    };
    auto solve = [&]() {
      int cl = col;
      asm volatile("" : "+v"(cl));
#pragma unroll
      for (int i = 0; i < kS; ++i) x[i] = (i == cl) ? 1.f : 0.f;
#pragma unroll
      for (int q = 0; q < kS; ++q) {
        if (q == 6 || q == 14) pbar(n);                // phases 4 and 5 start here
        if (q + 2 < kS) load_col(q + 2, cb[(q + 2) % 3]);
        const float xq = x[q];
        const float4* cv = cb[q % 3];
#pragma unroll
        for (int i = q + 1; i < kS; ++i) {
          const float4 v = cv[i / 4];
          const float aiq = (i & 3) == 0 ? v.x : (i & 3) == 1 ? v.y : (i & 3) == 2 ? v.z : v.w;
          x[i] = fmaf(-aiq, xq, x[i]);
        }
#pragma unroll
        for (int i = q + 1; i < kS; ++i) asm volatile("" : "+v"(x[i]));
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    // phase 6: Tu^T and Tw^T rows (columns of T diag(beta) and
    // T diag(beta 2^G), each rounded once; lane `col` writes row `col`), Tu
    // into the shared ring, Tw into the private area (A is no longer read)
    auto pack = [&](int m) {
      const float bc = gsc_l[kS + col];
      const float wc = bc * exp2f(gsc_l[col]);
      lchar* Tu = tubuf(m + hc);
      lchar* Tw = priv + hc * CF::SZ_TT;
#pragma unroll
      for (int q = 0; q < kS / 8; ++q) {
        // Tu in two bf16 parts (hi + lo): U = Tu V is the state's only
        // product whose rounding does not average over the segment
        uint32_t th[4], tl[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float u0 = x[8 * q + 2 * e] * bc, u1 = x[8 * q + 2 * e + 1] * bc;
          th[e] = pack_bf16x2(u0, u1);
          tl[e] = pack_bf16x2(u0 - bf16_bits_to_f32((uint16_t)th[e]), u1 - __uint_as_float(th[e] & 0xffff0000u));
        }
        uint4 tw;
        tw.x = pack_bf16x2(x[8 * q + 0] * wc, x[8 * q + 1] * wc);
        tw.y = pack_bf16x2(x[8 * q + 2] * wc, x[8 * q + 3] * wc);
        tw.z = pack_bf16x2(x[8 * q + 4] * wc, x[8 * q + 5] * wc);
        tw.w = pack_bf16x2(x[8 * q + 6] * wc, x[8 * q + 7] * wc);
        lds_st16(Tu + (col * kTP + 8 * q) * 2, make_uint4(th[0], th[1], th[2], th[3]));
        lds_st16(Tu + CF::SZ_TT + (col * kTP + 8 * q) * 2, make_uint4(tl[0], tl[1], tl[2], tl[3]));
        lds_st16(Tw + (col * kTP + 8 * q) * 2, tw);
      }
    };
    // phases 7 and 0: W^T = K^T Tw^T for sub-chunk m + c: lane (li, g) of
    // tile (td, bi) ends with W[16 bi + li][16 td + 4g ..], stored negated
    // (the state subtracts W M0) as an 8-byte row-major store
    auto make_w = [&](int mc, int c) {
      const lchar* Tw = priv + c * CF::SZ_TT;
      const lchar* Kc = kbuf(mc);
      lchar* Wc = wbuf(mc);
      // every read first: the compiler cannot move them above the W stores
      const bf16x8 tw0 = tr_pair(Tw + tr_t, kTP * 2, false);
      const bf16x8 tw1 = tr_pair(Tw + tr_t + 16 * 2, kTP * 2, false);
      bf16x8 kt[NT];
#pragma unroll
      for (int td = 0; td < NT; ++td) kt[td] = tr_kv(Kc, td);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int h = 0; h < NT; h += 4) {
        f32x4 w0[4], w1[4];
#pragma unroll
        for (int e = 0; e < 4 && h + e < NT; ++e) {
          w0[e] = mma_k32(zero4(), kt[h + e], tw0);
          w1[e] = mma_k32(zero4(), kt[h + e], tw1);
        }
#pragma unroll
        for (int e = 0; e < 4 && h + e < NT; ++e) {
          const int td = h + e;
          const int pos = 32 * (td >> 1) + 4 * (td & 1);   // column 16 td + 4g .. stored at 32 (td/2) + 8g + 4 (td%2)
          lds_st8(Wc + w_row + pos * 2, make_uint2(pack_bf16x2(-w0[e][0], -w0[e][1]), pack_bf16x2(-w0[e][2], -w0[e][3])));
          lds_st8(Wc + w_row + (16 * WP + pos) * 2, make_uint2(pack_bf16x2(-w1[e][0], -w1[e][1]), pack_bf16x2(-w1[e][2], -w1[e][3])));
        }
      }
    };

    // steps -9 .. NSC-1, one barrier each: pair m runs phase s at step
    // m - 9 + s, and phase 0 also finishes the previous pair
    while (n < 2 * p - 9 && n < NSC) {
      dma_duty(n);
      pbar(n);
    }
    int m = 2 * p;
    if (m < NSC) issue_loads(m);
    for (; m < NSC; m += 8) {
      if (m >= 8) make_w(m - 7, 1);            // m - 7 < NSC: the previous pair's second sub-chunk
      pbar(n);
      gram(m);
      dma_duty(n);                             // after the Gram fragments' loads were waited for
      pbar(n);
      make_a();
      load_col(0, cb[0]);                      // the solve's first columns (same wave: after the A stores)
      load_col(1, cb[1]);
      dma_duty(n);
      pbar(n);
      solve();                                 // phases 3, 4 and 5 (two barriers inside)
      pbar(n);
      pack(m);
      pbar(n);
      make_w(m, 0);
      if (m + 8 < NSC) issue_loads(m + 8);     // two steps before its Gram
      pbar(n);
    }
    if (m >= 8 && m - 7 < NSC) {                 // the last pair's second sub-chunk, at step m - 9
      make_w(m - 7, 1);
      dma_duty(n);
      pbar(n);
    }
    while (n < NSC) {
      dma_duty(n);
      pbar(n);
    }
    return;
  }

  // ================================================================== state
  // tile (td, cc) holds M[16 td + 4g + r][32 sw + 16 cc + li]
  const int sw = wid - NP;
  f32x4 M[NT][2];

  // The operands of a state step, read one step ahead: during step n the
  // wave issues the MFMAs of sub-chunk n from registers, then reads
  // sub-chunk n+1's operands, whose latency overlaps those MFMAs and the
  // barrier.
  bf16x8 t0, t1, t0l, t1l, vf[2], wf[NT / 2][2], kt[NT];
  float4 e0, e1;
  float decay;
  auto load_ops = [&](int m) {
    const lchar* Kc = kbuf(m);
    const lchar* Vc = vbuf(m);
    const lchar* Wc = wbuf(m);
    const lchar* Tu = tubuf(m);
    const SR_LDS float* vec = vecbuf(m);
    t0 = tr_pair(Tu + tr_t, kTP * 2, false);
    t1 = tr_pair(Tu + tr_t + 16 * 2, kTP * 2, false);
    t0l = tr_pair(Tu + CF::SZ_TT + tr_t, kTP * 2, false);
    t1l = tr_pair(Tu + CF::SZ_TT + tr_t + 16 * 2, kTP * 2, false);
#pragma unroll
    for (int cc = 0; cc < 2; ++cc) vf[cc] = tr_kv(Vc, 2 * sw + cc);
    // W rows 16 bi + li in the state's k order (stored that way)
#pragma unroll
    for (int q = 0; q < NT / 2; ++q)
#pragma unroll
      for (int bi = 0; bi < 2; ++bi) wf[q][bi] = as_bf16x8(lds_ld16(Wc + w_row + (16 * bi * WP + 32 * q) * 2));
    e0 = lds_ldf4((const lchar*)(vec + 4 * g));
    e1 = lds_ldf4((const lchar*)(vec + 16 + 4 * g));
    decay = vec[kS];
#pragma unroll
    for (int td = 0; td < NT; ++td) kt[td] = tr_kv(Kc, td);
  };
  // The state lines of a sub-chunk for this wave's 32 columns, in six phases
  // that pair each group of MFMAs with VALU work it does not wait on: the
  // two column tiles cc run one after the other, so the bf16 copies of the
  // state, its decay and the scaled Delta of one tile are formed under the
  // other tile's products.  Each accumulator sees its products in the same
  // order as a plain loop would give them, so the results do not depend on
  // this schedule.
  auto state_step = [&]() {
    f32x4 dl[2][2];
    bf16x8 mb[NT / 2], dfr[2];
    // U = Tu V for row halves bi of column tile cc (the bf16 copy of M0's
    // tile cc made under those products)
    auto u_and_copy = [&](int cc) {
      dl[0][cc] = mma_k32(mma_k32(zero4(), t0l, vf[cc]), t0, vf[cc]);
      dl[1][cc] = mma_k32(mma_k32(zero4(), t1l, vf[cc]), t1, vf[cc]);
#pragma unroll
      for (int q = 0; q < NT / 2; ++q) mb[q] = acc_pair(M[2 * q][cc], M[2 * q + 1][cc]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, NT / 2, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    };
    // Delta = U + (-W) M0 for column tile cc
    auto wm = [&](int cc) {
#pragma unroll
      for (int q = 0; q < NT / 2; ++q)
#pragma unroll
        for (int bi = 0; bi < 2; ++bi) dl[bi][cc] = mma_k32(dl[bi][cc], wf[q][bi], mb[q]);
    };
    // M's tile cc decays once its bf16 copy is made
    auto decay_tile = [&](int cc, int td0, int td1) {
#pragma unroll
      for (int td = td0; td < td1; ++td)
#pragma unroll
        for (int r = 0; r < 4; ++r) M[td][cc][r] *= decay;
    };
    // rows scaled by 2^{G_31 - G_i}, as the bf16 operand of M += K^T Delta
    auto scale_delta = [&](int cc) {
      dfr[cc] = as_bf16x8(make_uint4(pack_bf16x2(dl[0][cc][0] * e0.x, dl[0][cc][1] * e0.y),
                                     pack_bf16x2(dl[0][cc][2] * e0.z, dl[0][cc][3] * e0.w),
                                     pack_bf16x2(dl[1][cc][0] * e1.x, dl[1][cc][1] * e1.y),
                                     pack_bf16x2(dl[1][cc][2] * e1.z, dl[1][cc][3] * e1.w)));
    };
    auto update = [&](int cc) {
#pragma unroll
      for (int td = 0; td < NT; ++td) M[td][cc] = mma_k32(M[td][cc], kt[td], dfr[cc]);
    };
    // NT MFMAs, each followed by up to 4 VALU instructions
    auto pair_groups = [&]() {
#pragma unroll
      for (int i = 0; i < NT; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    };
    u_and_copy(0);                       // 1: U of tile 0 | bf16 copy of M0's tile 0
    wm(0);                               // 2: (-W) M0 into tile 0 | decay of M's tile 0
    decay_tile(0, 0, NT);
    pair_groups();
    u_and_copy(1);                       // 3: U of tile 1 | bf16 copy of M0's tile 1
    wm(1);                               // 4: (-W) M0 into tile 1 | scaled Delta of tile 0, half the decay of tile 1
    scale_delta(0);
    decay_tile(1, 0, NT / 2);
    pair_groups();
    update(0);                           // 5: M += K^T Delta for tile 0 | the rest, scaled Delta of tile 1
    decay_tile(1, NT / 2, NT);
    scale_delta(1);
    pair_groups();
    update(1);                           // 6: M += K^T Delta for tile 1
  };

  // ---- steps -9 .. NSC-1: the state lines of sub-chunk n, then the reads
  // of sub-chunk n+1's operands (K and V arrive by the prep waves' DMAs).
  // A unit's state starts at its first sub-chunk from zero (or its initial
  // state) and is stored after its last one.
  Cursor cs = cursor_new();   // unit of sub-chunk n
  auto unit_base = [&](const Cursor& c) {
    return state_base(uni(u_slot[c.k]), uni(u_lh[c.k]) % a.H_v) + (size_t)(4 * g) * spitch + 32 * sw + li;
  };
  // this lane's state element (16 td + r, 16 cc) of the wave's columns lies
  // inside the unit's rows and columns
  auto in_state = [&](int td, int cc, int r) { return 4 * g + 16 * td + r < srows && 32 * sw + li + 16 * cc < scols; };
  for (int n = -9; n < NSC; ++n) {
    if (n >= 0) {
      if (n >= cs.end) (void)sub(n, cs);
      if (n == cs.beg) {
        const float* si = st_in_of(uni(u_lh[cs.k]) / a.H_v);
        const size_t base = unit_base(cs);
#pragma unroll
        for (int td = 0; td < NT; ++td)
#pragma unroll
          for (int cc = 0; cc < 2; ++cc)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              M[td][cc][r] = si && in_state(td, cc, r) ? si[base + (size_t)(16 * td + r) * spitch + 16 * cc] : 0.f;
      }
      state_step();
      if (n + 1 == cs.end) {
        float* out = st_out_of(uni(u_lh[cs.k]) / a.H_v) + unit_base(cs);
#pragma unroll
        for (int td = 0; td < NT; ++td)
#pragma unroll
          for (int cc = 0; cc < 2; ++cc)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (in_state(td, cc, r)) out[(size_t)(16 * td + r) * spitch + 16 * cc] = M[td][cc][r];
      }
    }
    if (n + 1 >= 0 && n + 1 < NSC) load_ops(n + 1);
    lds_barrier();
  }
}

// Compute units of the current device (one workgroup fits per CU).
int device_cus() {
  static int cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cache[dev] = n;
  }
  return cache[dev];
}

template <int D, bool SPLIT = false>
hipError_t run(const ScanArgs& a, hipStream_t s) {
  const int64_t units = (int64_t)a.n_seg * a.n_layers * a.H_v;
  if (units == 0) return hipSuccess;
  // one workgroup per CU, each running its share of the units back to back
  // (at most kScanUnits)
  int64_t grid = units < device_cus() ? units : device_cus();
  if (grid * kScanUnits < units) grid = (units + kScanUnits - 1) / kScanUnits;
  hipLaunchKernelGGL((gdn_scan_bf16_kernel<D, SPLIT>), dim3((unsigned)grid), dim3(Cfg<D>::THREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_scan_bf16(int d_head, const ScanArgs& a, hipStream_t s) {
  if (a.v_split > 1) {
    // value heads split into units of 128 state columns (rectangular heads)
    if (d_head != 128 || a.H_v % a.v_split || a.st_rows <= 0 || a.st_rows > 128 || a.st_cols <= 0 ||
        a.st_cols > 128 || a.st_pitch < a.v_split * a.st_cols)
      return hipErrorInvalidValue;
    return run<128, true>(a, s);
  }
  switch (d_head) {
    case 32: return run<32>(a, s);
    case 64: return run<64>(a, s);
    case 128: return run<128>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace sr
