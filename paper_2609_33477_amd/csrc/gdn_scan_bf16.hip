// Chunked Gated DeltaNet state accumulation, bf16 operands (gfx950).
//
// Same recurrence as the fp32 kernel (gdn_scan.hip).  Rows go 64 at a time
// (a chunk) as four 16-row sub-chunks b; within a sub-chunk that starts from
// state M0 (= S^T), with G the sub-chunk prefix of log alpha:
//   A_ij  = beta_i e^{G_i - G_j} k_i.k_j  (i > j)        T = (I + A)^{-1}  (16x16)
//   U     = T diag(beta) V,    W = T diag(beta e^G) K
//   Delta = U - W M0
//   M_16  = e^{G_15} M0 + K^T diag(e^{G_15 - G}) Delta
// Only the last two lines touch the state.  The workgroup is split in two
// roles that run one chunk apart:
//   prep waves (4, one per sub-chunk) build T, Tu = T diag(beta) and W for
//     chunk c+1 -- Gram block, gates, a 16x16 forward substitution, one
//     16x16xd product;
//   state waves (d/16, wave s owning state columns [16s, 16s+16) as d/16
//     16x16 fp32 accumulator tiles) form U for their columns, run the four
//     state steps of chunk c back to back in registers, and stage the rows
//     of chunks c+2 (K) and c+1 (V) from registers loaded a step earlier.
// So per chunk the serial path is the state steps alone; the triangular
// solves of the next chunk overlap them.  Two barriers per chunk hand the
// double-buffered K, W, Tu and gate vectors from one role to the other.
//
// Products use v_mfma_f32_16x16x32_bf16 (reduction over d) and
// v_mfma_f32_16x16x16_bf16 (reduction over a sub-chunk's 16 rows).  K and V
// stay row-major in LDS; operands whose reduction index runs down the rows of
// an LDS matrix are read with ds_read_b64_tr_b16, which hands lane i of each
// 16-lane group rows kbase..kbase+3 of column n0 + i when lane j of the group
// addresses row kbase + j/4, columns n0 + 4 (j%4) .. +3.  W M0 takes the state
// straight from accumulator registers, with the MFMA k slots permuted to the
// accumulator row order and W read in the same order.
//
// LDS (d = 128): K x2, V, W^T x2 (~18 KB each), A 5 KB, Tu x2 | Tw 8 KB,
// vectors 2 KB: ~105 KB, one workgroup (12 waves) per CU.
#include "sr_device.hpp"

#include <cstddef>

namespace sr {
namespace {

constexpr int kC = 64;       // rows staged per step
constexpr int kS = 16;       // sub-chunk rows
constexpr int kAP = 20;      // fp32 pitch of the 16x16 A blocks
constexpr int kTP = 20;      // bf16 pitch of the 16x16 Tu / Tw blocks
constexpr int kSortMax = 256;

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
__device__ __forceinline__ void lds_st8(lchar* p, const uint2& v) {
  *reinterpret_cast<SR_LDS nu32x2*>(p) = __builtin_bit_cast(nu32x2, v);
}

// Transposed read (see the file comment); `p` includes the lane part of the
// address.
__device__ __forceinline__ uint2 tr4(const lchar* p) {
  const v4i16 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((SR_LDS v4i16*)p);
  return __builtin_bit_cast(uint2, v);
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
  static constexpr int NS = D / 16;                   // state waves; wave s owns columns [16s, 16s+16)
  static constexpr int NP = 4;                        // prep waves, one per sub-chunk
  static constexpr int THREADS = 64 * (NS + NP);
  static constexpr int NT = D / 16;                   // 16-row tiles along d
  static constexpr int KP = D + 16;                   // K / V row pitch (bf16): conflict-free 16-byte and
                                                      // transposed reads
  static constexpr int WP = kC + 8;                   // W^T row pitch (bf16)
  static constexpr int SZ_KV = kC * KP * 2;
  static constexpr int SZ_W = D * WP * 2;
  static constexpr int SZ_TU = kC * kTP * 2;          // Tu of one chunk (four 16x16 bf16 blocks)
  static constexpr int SZ_TW = kS * kTP * 2;          // Tw of one sub-chunk (prep-wave private)
  static constexpr int SZ_A = kS * kAP * 4;           // A of one sub-chunk (prep-wave private)
  static constexpr int SZ_VEC = 2 * kC * 4;           // eG | eD of one chunk
  static constexpr int SZ_SCR = 2 * kS * 4;           // G prefix | beta of one sub-chunk (prep-wave private)
  static constexpr int OFF_K = 0;                     // two K buffers
  static constexpr int OFF_V = OFF_K + 2 * SZ_KV;
  static constexpr int OFF_W = OFF_V + SZ_KV;         // two W^T buffers
  static constexpr int OFF_TU = OFF_W + 2 * SZ_W;     // two Tu buffers
  static constexpr int OFF_TW = OFF_TU + 2 * SZ_TU;
  static constexpr int OFF_A = OFF_TW + NP * SZ_TW;
  static constexpr int OFF_VEC = OFF_A + NP * SZ_A;   // two vector buffers
  static constexpr int OFF_SCR = OFF_VEC + 2 * SZ_VEC;
  static constexpr int LDS = OFF_SCR + NP * SZ_SCR;
  static constexpr int PPR = D / 8;                   // 16-byte pieces per row
  static constexpr int PER_S = kC * PPR / (64 * NS);  // pieces per state thread per matrix (2)
  static_assert(kC * PPR % (64 * NS) == 0, "staging split");
};

__device__ int rank_to_segment(const ScanArgs& a, int rank, int* shared_sel) {
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

template <int D>
__global__ __launch_bounds__(64 * (D / 16 + 4), 1) void gdn_scan_bf16_kernel(ScanArgs a) {
  using CF = Cfg<D>;
  constexpr int NS = CF::NS, NP = CF::NP, NT = CF::NT, KP = CF::KP, WP = CF::WP;
  __shared__ __attribute__((aligned(16))) char smem[CF::LDS];
  __shared__ int sel;

  lchar* L = (lchar*)smem;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, li = lane & 15;
  // per-lane byte offsets; everything else is a compile-time immediate
  const int kv_row = (li * KP + 8 * g) * 2;                           // 16-byte row reads of K
  const int t_row = (li * kTP + 4 * g) * 2;                           // 8-byte row reads of Tu / Tw
  const int tr_kv = ((li >> 2) * KP + 4 * (li & 3) + 4 * g * KP) * 2; // transposed reads of K / V, rows 4g + ..
  const int tr_w = ((li >> 2) * WP + 4 * (li & 3) + 4 * g * WP) * 2;  // transposed reads of W^T, rows 4g + ..

  const int u = blockIdx.x;
  const int head = u % a.H_v;
  const int layer = (u / a.H_v) % a.n_layers;
  const int rank = u / (a.H_v * a.n_layers);
  const int b = rank_to_segment(a, rank, &sel);
  const int slot = a.slot_ids ? a.slot_ids[b] : b;
  if (slot < 0) return;
  const int64_t s0 = a.cu[b], s1 = a.cu[b + 1];
  const int nch = (int)((s1 - s0 + kC - 1) / kC);
  const int hk = (head * a.H_k) / a.H_v;

  const char* Kplane = static_cast<const char*>(a.Kbuf) + (layer * a.k_layer_stride + (int64_t)hk * a.T * D) * 2;
  const char* Vplane = static_cast<const char*>(a.Vbuf) + (layer * a.v_layer_stride + (int64_t)head * a.T * D) * 2;
  const float* Gp = a.Gbuf + layer * a.g_layer_stride + (int64_t)head * a.T;
  const float* Bp = a.Bbuf + layer * a.g_layer_stride + (int64_t)head * a.T;
  // Per-layer state pointers from the kernel-argument segment at a uniform
  // offset (ScanArgs is the only argument, at offset 0).
  const char* kargs = (const char*)__builtin_amdgcn_kernarg_segment_ptr();
  const float* st_in = *reinterpret_cast<const float* const*>(kargs + offsetof(ScanArgs, state_in) + sizeof(void*) * layer);
  float* st_out = *reinterpret_cast<float* const*>(kargs + offsetof(ScanArgs, state_out) + sizeof(void*) * layer);
  const size_t state_base = ((size_t)slot * a.H_v + head) * D * D;

  auto kbuf = [&](int c) { return L + CF::OFF_K + (c & 1) * CF::SZ_KV; };
  auto wbuf = [&](int c) { return L + CF::OFF_W + (c & 1) * CF::SZ_W; };
  auto tubuf = [&](int c) { return L + CF::OFF_TU + (c & 1) * CF::SZ_TU; };
  auto vecbuf = [&](int c) { return (SR_LDS float*)(L + CF::OFF_VEC + (c & 1) * CF::SZ_VEC); };  // eG[64] | eD[64]
  lchar* Vr = L + CF::OFF_V;

  const bool prep = wid < NP;
  // ---- prep-wave state
  const int sb = prep ? wid : 0;                         // sub-chunk of a prep wave
  lchar* Tw = L + CF::OFF_TW + sb * CF::SZ_TW;
  SR_LDS float* Am = (SR_LDS float*)(L + CF::OFF_A + sb * CF::SZ_A);
  SR_LDS float* gsc = (SR_LDS float*)(L + CF::OFF_SCR + sb * CF::SZ_SCR);   // G prefix [16] | beta [16]
  // ---- state-wave state: tile td holds M[16 td + 4g + r][16 s + li]; the
  // state waves also stage the K / V rows (prefetched a step ahead)
  const int sw = prep ? 0 : wid - NP;
  const int stid = tid - 64 * NP;
  f32x4 M[NT];
  uint4 pk[CF::PER_S], pv[CF::PER_S];

  // rows of chunk c as 16-byte pieces (zero past the segment end)
  auto load_rows = [&](const char* plane, int c, uint4* dst) {
    const int64_t c0 = s0 + (int64_t)c * kC;
#pragma unroll
    for (int i = 0; i < CF::PER_S; ++i) {
      const int p = stid + i * 64 * NS;
      const int row = p / CF::PPR, cc = p % CF::PPR;
      const int64_t t = c0 + row;
      dst[i] = (c < nch && t < s1) ? *reinterpret_cast<const uint4*>(plane + (t * D + cc * 8) * 2) : make_uint4(0, 0, 0, 0);
    }
  };
  auto store_rows = [&](lchar* buf, const uint4* src) {
#pragma unroll
    for (int i = 0; i < CF::PER_S; ++i) {
      const int p = stid + i * 64 * NS;
      const int row = p / CF::PPR, cc = p % CF::PPR;
      lds_st16(buf + (row * KP + cc * 8) * 2, src[i]);
    }
  };
  // log2 alpha and beta of sub-chunk sb's 16 rows of chunk c (lanes 0..15;
  // rows past the segment end carry 0 and 0, which makes them inert)
  auto load_gb = [&](int c, float& gv, float& bv) {
    const int64_t t = s0 + (int64_t)c * kC + 16 * sb + li;
    const bool ok = lane < 16 && c < nch && t < s1;
    gv = ok ? Gp[t] : 0.f;
    bv = ok ? Bp[t] : 0.f;
  };

  // prep: T, Tu, W and the gate vectors of sub-chunk sb of chunk c
  auto prep_chunk = [&](int c, float gv, float bv) {
    const lchar* Kc = kbuf(c);
    // inclusive prefix of log2 alpha over the 16 rows (lanes 0..15)
    float gp = gv;
    gp += dpp_row_shr<1>(gp);
    gp += dpp_row_shr<2>(gp);
    gp += dpp_row_shr<4>(gp);
    gp += dpp_row_shr<8>(gp);
    const float g15 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, gp), 15));
    SR_LDS float* vec = vecbuf(c);
    if (lane < 16) {
      gsc[li] = gp;
      gsc[16 + li] = bv;
      vec[16 * sb + li] = exp2f(gp);             // 2^{G_i}
      vec[kC + 16 * sb + li] = exp2f(g15 - gp);  // 2^{G_15 - G_i}
    }
    // Gram block and A = beta_i 2^{G_i - G_j} Gamma (i > j)
    f32x4 gam = zero4();
#pragma unroll
    for (int s = 0; s < D / 32; ++s) {
      const bf16x8 kf = as_bf16x8(lds_ld16(Kc + kv_row + (16 * sb * KP + 32 * s) * 2));
      gam = mma_k32(gam, kf, kf);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);          // this wave's writes of gsc have landed
    const float gj = gsc[li];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 4 * g + r;
      Am[i * kAP + li] = (i > li) ? gsc[16 + i] * exp2f(fminf(gsc[i] - gj, 0.f)) * gam[r] : 0.f;
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);
    // T = (I + A)^{-1} by forward substitution, lane = column (every 16-lane
    // group solves the same block; group 0 writes).  The column index goes
    // through an empty asm so the 16 identity selects stay inside the loop
    // instead of being hoisted into registers live across all chunks.
    int col = li;
    asm volatile("" : "+v"(col));
    float x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if (i % 4 == 0) __builtin_amdgcn_sched_barrier(0);   // bound the hoisting of A loads
      float t0 = (i == col) ? 1.f : 0.f, t1 = 0.f;
#pragma unroll
      for (int q = 0; q < (i + 3) / 4; ++q) {
        const float4 v = lds_ldf4((const lchar*)(Am + i * kAP + 4 * q));
        if (4 * q + 0 < i) t0 = fmaf(-v.x, x[4 * q + 0], t0);
        if (4 * q + 1 < i) t1 = fmaf(-v.y, x[4 * q + 1], t1);
        if (4 * q + 2 < i) t0 = fmaf(-v.z, x[4 * q + 2], t0);
        if (4 * q + 3 < i) t1 = fmaf(-v.w, x[4 * q + 3], t1);
      }
      x[i] = t0 + t1;
    }
    // Tu = T diag(beta), Tw = T diag(beta 2^G), each rounded once
    const float bc = gsc[16 + li];
    const float wc = bc * exp2f(gsc[li]);
    lchar* Tu = tubuf(c);
    if (lane < 16) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        *reinterpret_cast<SR_LDS uint16_t*>(Tu + ((16 * sb + i) * kTP + li) * 2) = f32_to_bf16_bits(x[i] * bc);
        *reinterpret_cast<SR_LDS uint16_t*>(Tw + (i * kTP + li) * 2) = f32_to_bf16_bits(x[i] * wc);
      }
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);
    // W = Tw K of this sub-chunk, stored as W^T
    lchar* Wt = wbuf(c);
    const v4i16 twf = as_v4(lds_ld8(Tw + t_row));
#pragma unroll
    for (int td = 0; td < NT; ++td) {
      const f32x4 w = mma_k16(zero4(), twf, as_v4(tr4(Kc + tr_kv + (16 * sb * KP + 16 * td) * 2)));
      lds_st8(Wt + ((16 * td + li) * WP + 16 * sb + 4 * g) * 2,
              make_uint2(pack_bf16x2(w[0], w[1]), pack_bf16x2(w[2], w[3])));
    }
  };

  // state: U for this wave's columns, then the four state steps of chunk c
  auto state_chunk = [&](int c) {
    const lchar* Kc = kbuf(c);
    const lchar* Tu = tubuf(c);
    const lchar* Wt = wbuf(c);
    const SR_LDS float* vec = vecbuf(c);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      // U for this sub-chunk and this wave's columns
      f32x4 dl = mma_k16(zero4(), as_v4(lds_ld8(Tu + t_row + 16 * s * kTP * 2)),
                         as_v4(tr4(Vr + tr_kv + (16 * s * KP + 16 * sw) * 2)));
#pragma unroll
      for (int p = 0; p < NT / 2; ++p)   // Delta = U - W M0, W rows read in the state's k order
        dl = mma_k32(dl,
                     join(tr4(Wt + tr_w + ((32 * p) * WP + 16 * s) * 2),
                          tr4(Wt + tr_w + ((32 * p + 16) * WP + 16 * s) * 2), true),
                     acc_pair(M[2 * p], M[2 * p + 1]));
      const float4 ed = lds_ldf4((const lchar*)(vec + kC + 16 * s + 4 * g));
      const v4i16 dfr = as_v4(make_uint2(pack_bf16x2(dl[0] * ed.x, dl[1] * ed.y), pack_bf16x2(dl[2] * ed.z, dl[3] * ed.w)));
      const float decay = vec[16 * s + 15];
#pragma unroll
      for (int td = 0; td < NT; ++td) {
#pragma unroll
        for (int r = 0; r < 4; ++r) M[td][r] *= decay;
        M[td] = mma_k16(M[td], as_v4(tr4(Kc + tr_kv + (16 * s * KP + 16 * td) * 2)), dfr);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // The two roles run separate loops (wave-uniform branch) so that neither
  // keeps the other's loop-invariant addresses live; both meet the same
  // sequence of barriers: two in the prologue and two per chunk.
  if (prep) {
    float g_nx = 0.f, b_nx = 0.f, g_pf = 0.f, b_pf = 0.f;
    if (nch > 0) {
      load_gb(1, g_nx, b_nx);
      load_gb(2, g_pf, b_pf);
    }
    lds_barrier();
    if (nch > 0) {
      float g0, b0;
      load_gb(0, g0, b0);
      prep_chunk(0, g0, b0);     // T / W of chunk 0
    }
    lds_barrier();
    for (int c = 0; c < nch; ++c) {
      if (c + 1 < nch) prep_chunk(c + 1, g_nx, b_nx);
      lds_barrier();
      g_nx = g_pf;
      b_nx = b_pf;
      load_gb(c + 3, g_pf, b_pf);
      lds_barrier();
    }
    return;
  }

  // ---- state waves.  Prologue: chunks 0 and 1 resident, the state loaded
  if (nch > 0) {
    load_rows(Kplane, 0, pk);
    load_rows(Vplane, 0, pv);
    store_rows(kbuf(0), pk);
    store_rows(Vr, pv);
    load_rows(Kplane, 1, pk);
    store_rows(kbuf(1), pk);
    load_rows(Kplane, 2, pk);       // K(2) -> K buffer 0 after step 0
    load_rows(Vplane, 1, pv);       // V(1) -> the V buffer after step 0
  }
#pragma unroll
  for (int td = 0; td < NT; ++td) {
    M[td] = zero4();
    if (st_in) {
#pragma unroll
      for (int r = 0; r < 4; ++r) M[td][r] = st_in[state_base + (size_t)(16 * td + 4 * g + r) * D + 16 * sw + li];
    }
  }
  lds_barrier();
  lds_barrier();

  // ---- pipeline: step c runs the state steps of chunk c while the prep
  // waves prepare c+1
  for (int c = 0; c < nch; ++c) {
    state_chunk(c);
    lds_barrier();
    if (c + 2 < nch) store_rows(kbuf(c), pk);
    if (c + 1 < nch) store_rows(Vr, pv);
    load_rows(Kplane, c + 3, pk);
    load_rows(Vplane, c + 2, pv);
    lds_barrier();
  }

  float* out = st_out + state_base;
#pragma unroll
  for (int td = 0; td < NT; ++td)
#pragma unroll
    for (int r = 0; r < 4; ++r) out[(size_t)(16 * td + 4 * g + r) * D + 16 * sw + li] = M[td][r];
}

template <int D>
hipError_t run(const ScanArgs& a, hipStream_t s) {
  const int64_t units = (int64_t)a.n_seg * a.n_layers * a.H_v;
  if (units == 0) return hipSuccess;
  hipLaunchKernelGGL((gdn_scan_bf16_kernel<D>), dim3((unsigned)units), dim3(Cfg<D>::THREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_scan_bf16(int d_head, const ScanArgs& a, hipStream_t s) {
  switch (d_head) {
    case 32: return run<32>(a, s);
    case 64: return run<64>(a, s);
    case 128: return run<128>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace sr
