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
//     sub-chunks m = p (mod 4), spread over the 4 steps before the state
//     needs them -- gates, Gram block and A (step m-4), a 32-step forward
//     substitution in fp32, lane = column of T (steps m-3 and m-2), then
//     Tu = T diag(beta) and W^T = K^T (T diag(beta 2^G))^T, which leaves W
//     row-major (step m-1);
//   d/32 state waves, wave s owning state columns [32s, 32s+32) as 2 d/16
//     16x16 fp32 accumulator tiles for the whole segment: at step m they
//     form U for their columns and run the state lines of sub-chunk m, and
//     they stage K five sub-chunks ahead and V one ahead from registers
//     loaded a step earlier.
// K lives in a ring of 6 sub-chunk slots, V, W and Tu in rings of 2.
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
// LDS (d = 128): K ring 54 KB, V and W rings 37 KB, Tu ring 6 KB, per prep
// wave A^T (reused for Tw^T) and gate scratch 19 KB: ~117 KB, one workgroup
// (8 waves) per CU.  Pitches are the measured conflict-free ones: row pitch
// = 8 mod 64 dwords for 16-byte row and transposed reads, 2 mod 8 dwords for
// 8-byte row reads and writes.
#include "sr_device.hpp"

#include <cstddef>

namespace sr {
namespace {

constexpr int kC = 64;       // rows staged per step
constexpr int kS = 32;       // sub-chunk rows
constexpr int kAP = 36;      // fp32 pitch of a sub-chunk's A (rows read as float4)
constexpr int kTP = 48;      // bf16 pitch of the T^T blocks (transposed reads)
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
__device__ __forceinline__ void lds_stf4(lchar* p, const float* v) {
  *reinterpret_cast<SR_LDS nf32x4*>(p) = nf32x4{v[0], v[1], v[2], v[3]};
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
  static constexpr int NSW = D / 32;                  // state waves; wave s owns columns [32s, 32s+32)
  static constexpr int NP = 4;                        // prep waves
  static constexpr int THREADS = 64 * (NSW + NP);
  static constexpr int NT = D / 16;                   // 16-row tiles along d
  static constexpr int KP = D + 16;                   // K / V row pitch (bf16)
  static constexpr int WP = D + 20;                   // W row pitch (bf16)
  static constexpr int NK = 6;                        // K ring slots
  static constexpr int SZ_KV = kS * KP * 2;           // one sub-chunk of K or V
  static constexpr int SZ_W = kS * WP * 2;
  static constexpr int SZ_TT = kS * kTP * 2;          // one T^T block (bf16)
  static constexpr int SZ_A = kS * kAP * 4;           // A^T of one sub-chunk (prep-wave private; later Tw^T)
  static constexpr int SZ_VEC = 2 * kS * 4;           // eG | eD of one sub-chunk
  static constexpr int SZ_SCR = 2 * kS * 4;           // G prefix | beta (prep-wave private)
  static constexpr int OFF_K = 0;
  static constexpr int OFF_V = OFF_K + NK * SZ_KV;
  static constexpr int OFF_W = OFF_V + 2 * SZ_KV;
  static constexpr int OFF_TU = OFF_W + 2 * SZ_W;
  static constexpr int OFF_A = OFF_TU + 4 * SZ_TT;     // two (Tu_hi^T | Tu_lo^T) slots
  static constexpr int OFF_VEC = OFF_A + NP * SZ_A;
  static constexpr int OFF_SCR = OFF_VEC + NK * SZ_VEC;
  static constexpr int LDS = OFF_SCR + NP * SZ_SCR;
  static constexpr int PPR = D / 8;                   // 16-byte pieces per row
  static constexpr int PER_S = kS * PPR / (64 * NSW); // pieces per state thread per matrix
  static constexpr int QS = 10;                       // solve steps in the first solve segment
  static_assert(kS * PPR % (64 * NSW) == 0, "staging split");
  static_assert(NT % 2 == 0, "state tiles pair up along d");
  static_assert(SZ_TT <= SZ_A, "Tw^T reuses the A^T area");
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
__global__ __launch_bounds__(64 * (D / 32 + 4), 1) void gdn_scan_bf16_kernel(ScanArgs a) {
  using CF = Cfg<D>;
  constexpr int NSW = CF::NSW, NP = CF::NP, NT = CF::NT, KP = CF::KP, WP = CF::WP, NK = CF::NK;
  __shared__ __attribute__((aligned(16))) char smem[CF::LDS];
  __shared__ int sel;

  lchar* L = (lchar*)smem;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, li = lane & 15;
  // per-lane byte offsets; everything else is a compile-time immediate
  const int kv_row = (li * KP + 8 * g) * 2;                           // 16-byte row reads of K
  const int w_row = (li * WP + 4 * g) * 2;                            // 8-byte row reads / writes of W
  const int tr_kv = ((li >> 2) * KP + 4 * (li & 3) + 4 * g * KP) * 2; // transposed reads of K / V, rows 4g + ..
  const int tr_t = ((li >> 2) * kTP + 4 * (li & 3) + 4 * g * kTP) * 2; // transposed reads of T^T, rows 4g + ..

  const int u = blockIdx.x;
  const int head = u % a.H_v;
  const int layer = (u / a.H_v) % a.n_layers;
  const int rank = u / (a.H_v * a.n_layers);
  const int b = rank_to_segment(a, rank, &sel);
  const int slot = a.slot_ids ? a.slot_ids[b] : b;
  if (slot < 0) return;
  const int64_t s0 = a.cu[b], s1 = a.cu[b + 1];
  const int nsc = (int)((s1 - s0 + kS - 1) / kS);     // sub-chunks
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

  auto kbuf = [&](int m) { return L + CF::OFF_K + (m % NK) * CF::SZ_KV; };
  auto vbuf = [&](int m) { return L + CF::OFF_V + (m & 1) * CF::SZ_KV; };
  auto wbuf = [&](int m) { return L + CF::OFF_W + (m & 1) * CF::SZ_W; };
  auto tubuf = [&](int m) { return L + CF::OFF_TU + (m & 1) * 2 * CF::SZ_TT; };   // Tu_hi^T, then Tu_lo^T
  auto vecbuf = [&](int m) { return (SR_LDS float*)(L + CF::OFF_VEC + (m % NK) * CF::SZ_VEC); };  // eG[32] | eD[32]

  // A 32-wide reduction operand from a transposed-read matrix: rows
  // kbase + {4g..4g+3} and kbase + 16 + {4g..4g+3} of the lane's column.
  auto tr_pair = [&](const lchar* p, int pitch_bytes, bool negate) {
    return join(tr4(p), tr4(p + 16 * pitch_bytes), negate);
  };

  if (wid < NP) {
    // ================================================================ prep
    const int p = wid;
    SR_LDS float* At = (SR_LDS float*)(L + CF::OFF_A + p * CF::SZ_A);   // A^T, later Tw^T (private)
    lchar* Tw = (lchar*)At;
    SR_LDS float* gsc = (SR_LDS float*)(L + CF::OFF_SCR + p * CF::SZ_SCR);   // G prefix [32] | beta [32]
    const int col = lane & 31;                           // column of T this lane solves

    // log2 alpha and beta of sub-chunk m's 32 rows (lanes 0..31; rows past
    // the segment end carry 0 and 0, which makes them inert)
    auto load_gb = [&](int m, float& gv, float& bv) {
      const int64_t t = s0 + (int64_t)m * kS + col;
      const bool ok = lane < 32 && m < nsc && t < s1;
      gv = ok ? Gp[t] : 0.f;
      bv = ok ? Bp[t] : 0.f;
    };

    float x[kS];                                         // column `col` of T, carried across segments
    // S1: prefix, gate vectors, Gram block, A^T
    auto seg_a = [&](int m, float gv, float bv) {
      const lchar* Kc = kbuf(m);
      float gp = gv;
      gp += dpp_row_shr<1>(gp);
      gp += dpp_row_shr<2>(gp);
      gp += dpp_row_shr<4>(gp);
      gp += dpp_row_shr<8>(gp);
      const float g15 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, gp), 15));
      if (lane >= 16) gp += g15;
      const float g31 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, gp), 31));
      SR_LDS float* vec = vecbuf(m);
      if (lane < 32) {
        gsc[col] = gp;
        gsc[kS + col] = bv;
        vec[col] = exp2f(gp);                 // 2^{G_i}
        vec[kS + col] = exp2f(g31 - gp);      // 2^{G_31 - G_i}
      }
      f32x4 g00 = zero4(), g10 = zero4(), g11 = zero4();
#pragma unroll
      for (int q = 0; q < D / 32; ++q) {
        const bf16x8 k0 = as_bf16x8(lds_ld16(Kc + kv_row + 32 * q * 2));
        const bf16x8 k1 = as_bf16x8(lds_ld16(Kc + kv_row + (16 * KP + 32 * q) * 2));
        g00 = mma_k32(g00, k0, k0);
        g10 = mma_k32(g10, k1, k0);
        g11 = mma_k32(g11, k1, k1);
      }
      __builtin_amdgcn_s_waitcnt(0xc07f);          // this wave's writes of gsc have landed
      const float gj0 = gsc[li], gj1 = gsc[16 + li];
      float a00[4], a10[4], a11[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i0 = 4 * g + r, i1 = 16 + 4 * g + r;
        const float b0 = gsc[kS + i0], b1 = gsc[kS + i1], gi0 = gsc[i0], gi1 = gsc[i1];
        a00[r] = (i0 > li) ? b0 * exp2f(fminf(gi0 - gj0, 0.f)) * g00[r] : 0.f;
        a10[r] = b1 * exp2f(fminf(gi1 - gj0, 0.f)) * g10[r];
        a11[r] = (i1 > 16 + li) ? b1 * exp2f(fminf(gi1 - gj1, 0.f)) * g11[r] : 0.f;
      }
      // stored transposed, At[j][i] = A_ij: one 16-byte store per block
      lds_stf4((lchar*)(At + li * kAP + 4 * g), a00);
      lds_stf4((lchar*)(At + li * kAP + 16 + 4 * g), a10);
      lds_stf4((lchar*)(At + (16 + li) * kAP + 16 + 4 * g), a11);
    };
    // S2 / S3: T = (I + A)^{-1}, lane = column, column-oriented: once
    // x_q = T[q][col] is final it is eliminated from every later row.  Each
    // step needs one column of A (a row of A^T), read two steps ahead; the
    // empty asm keeps each step's updates in place (later loads may not be
    // hoisted above them, nor the updates sunk below).
    auto solve = [&](auto q0_tag, auto q1_tag) {
      constexpr int Q0 = decltype(q0_tag)::value, Q1 = decltype(q1_tag)::value;
      float4 cb[3][kS / 4];
      auto load_col = [&](int q, float4* dst) {
#pragma unroll
        for (int v = (q + 1) / 4; v < kS / 4; ++v) dst[v] = lds_ldf4((const lchar*)(At + q * kAP + 4 * v));
      };
      load_col(Q0, cb[Q0 % 3]);
      if (Q0 + 1 < Q1) load_col(Q0 + 1, cb[(Q0 + 1) % 3]);
#pragma unroll
      for (int q = Q0; q < Q1; ++q) {
        if (q + 2 < Q1) load_col(q + 2, cb[(q + 2) % 3]);
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
    // S4: Tu^T and Tw^T rows (columns of T diag(beta) and T diag(beta 2^G),
    // each rounded once; lane `col` writes row `col`), then W^T = K^T Tw^T:
    // lane (li, g) of tile (td, bi) ends with W[16 bi + li][16 td + 4g ..],
    // stored negated (the state subtracts W M0) as an 8-byte row-major store
    auto seg_d = [&](int m) {
      const float bc = gsc[kS + col];
      const float wc = bc * exp2f(gsc[col]);
      lchar* Tu = tubuf(m);
      if (lane < 32) {
#pragma unroll
        for (int q = 0; q < kS / 8; ++q) {
          // Tu in two bf16 parts (hi + lo): U = Tu V is the state's only
          // product whose rounding does not average over the segment
          uint32_t th[4], tl[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float u0 = x[8 * q + 2 * e] * bc, u1 = x[8 * q + 2 * e + 1] * bc;
            th[e] = pack_bf16x2(u0, u1);
            tl[e] = pack_bf16x2(u0 - bf16_bits_to_f32((uint16_t)th[e]), u1 - bf16_bits_to_f32((uint16_t)(th[e] >> 16)));
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
      }
      __builtin_amdgcn_s_waitcnt(0xc07f);
      const lchar* Kc = kbuf(m);
      lchar* Wc = wbuf(m);
      const bf16x8 tw0 = tr_pair(Tw + tr_t, kTP * 2, false);
      const bf16x8 tw1 = tr_pair(Tw + tr_t + 16 * 2, kTP * 2, false);
#pragma unroll
      for (int td = 0; td < NT; ++td) {
        const bf16x8 kt = tr_pair(Kc + tr_kv + 16 * td * 2, KP * 2, false);
        const f32x4 w0 = mma_k32(zero4(), kt, tw0);
        const f32x4 w1 = mma_k32(zero4(), kt, tw1);
        lds_st8(Wc + w_row + 16 * td * 2, make_uint2(pack_bf16x2(-w0[0], -w0[1]), pack_bf16x2(-w0[2], -w0[3])));
        lds_st8(Wc + w_row + (16 * WP + 16 * td) * 2, make_uint2(pack_bf16x2(-w1[0], -w1[1]), pack_bf16x2(-w1[2], -w1[3])));
      }
    };

    // after the barrier that publishes K(0): steps -4 .. nsc-1, one barrier
    // each; this wave runs sub-chunks
    // m = p, p + 4, ... in steps m-4 .. m-1
    lds_barrier();                                       // K(0) is in place
    int n = -4;
    for (; n < p - 4; ++n) lds_barrier();
    float gv, bv, gv_nx, bv_nx;
    load_gb(p, gv, bv);
    for (int m = p; m < nsc; m += 4) {
      load_gb(m + 4, gv_nx, bv_nx);
      seg_a(m, gv, bv);
      lds_barrier();
      int cl = col;
      asm volatile("" : "+v"(cl));
#pragma unroll
      for (int i = 0; i < kS; ++i) x[i] = (i == cl) ? 1.f : 0.f;
      solve(std::integral_constant<int, 0>{}, std::integral_constant<int, CF::QS>{});
      lds_barrier();
      solve(std::integral_constant<int, CF::QS>{}, std::integral_constant<int, kS>{});
      lds_barrier();
      seg_d(m);
      lds_barrier();
      gv = gv_nx;
      bv = bv_nx;
      n += 4;
    }
    for (; n < nsc; ++n) lds_barrier();
    return;
  }

  // ================================================================== state
  // tile (td, cc) holds M[16 td + 4g + r][32 sw + 16 cc + li]
  const int sw = wid - NP;
  const int stid = tid - 64 * NP;
  f32x4 M[NT][2];
  uint4 pk[CF::PER_S], pv[CF::PER_S];

  // rows of sub-chunk m as 16-byte pieces (zero past the segment end)
  auto load_rows = [&](const char* plane, int m, uint4* dst) {
    const int64_t c0 = s0 + (int64_t)m * kS;
#pragma unroll
    for (int i = 0; i < CF::PER_S; ++i) {
      const int q = stid + i * 64 * NSW;
      const int row = q / CF::PPR, cc = q % CF::PPR;
      const int64_t t = c0 + row;
      dst[i] = (m >= 0 && m < nsc && t < s1) ? *reinterpret_cast<const uint4*>(plane + (t * D + cc * 8) * 2)
                                             : make_uint4(0, 0, 0, 0);
    }
  };
  auto store_rows = [&](lchar* buf, const uint4* src) {
#pragma unroll
    for (int i = 0; i < CF::PER_S; ++i) {
      const int q = stid + i * 64 * NSW;
      const int row = q / CF::PPR, cc = q % CF::PPR;
      lds_st16(buf + (row * KP + cc * 8) * 2, src[i]);
    }
  };

  // the state lines of sub-chunk m for this wave's 32 columns.  Every LDS
  // read of the step is issued first, so their latencies overlap instead of
  // each one stalling the MFMA that needs it.
  auto state_step = [&](int m) {
    const lchar* Kc = kbuf(m);
    const lchar* Vc = vbuf(m);
    const lchar* Wc = wbuf(m);
    const lchar* Tu = tubuf(m);
    const SR_LDS float* vec = vecbuf(m);
    const bf16x8 t0 = tr_pair(Tu + tr_t, kTP * 2, false);
    const bf16x8 t1 = tr_pair(Tu + tr_t + 16 * 2, kTP * 2, false);
    const bf16x8 t0l = tr_pair(Tu + CF::SZ_TT + tr_t, kTP * 2, false);
    const bf16x8 t1l = tr_pair(Tu + CF::SZ_TT + tr_t + 16 * 2, kTP * 2, false);
    bf16x8 vf[2], wf[NT / 2][2], kt[NT];
#pragma unroll
    for (int cc = 0; cc < 2; ++cc) vf[cc] = tr_pair(Vc + tr_kv + (32 * sw + 16 * cc) * 2, KP * 2, false);
#pragma unroll
    for (int q = 0; q < NT / 2; ++q)
#pragma unroll
      for (int bi = 0; bi < 2; ++bi) {
        const lchar* wr = Wc + w_row + (16 * bi * WP + 32 * q) * 2;
        wf[q][bi] = join(lds_ld8(wr), lds_ld8(wr + 16 * 2), false);
      }
    const float4 e0 = lds_ldf4((const lchar*)(vec + kS + 4 * g));
    const float4 e1 = lds_ldf4((const lchar*)(vec + kS + 16 + 4 * g));
    const float decay = vec[kS - 1];
#pragma unroll
    for (int td = 0; td < NT; ++td) kt[td] = tr_pair(Kc + tr_kv + 16 * td * 2, KP * 2, false);
    __builtin_amdgcn_sched_barrier(0);
    // U = Tu V for row halves bi and column tiles cc; Delta = U + (-W) M0,
    // W rows read in the state's k order
    f32x4 dl[2][2];
#pragma unroll
    for (int cc = 0; cc < 2; ++cc) {
      dl[0][cc] = mma_k32(mma_k32(zero4(), t0l, vf[cc]), t0, vf[cc]);
      dl[1][cc] = mma_k32(mma_k32(zero4(), t1l, vf[cc]), t1, vf[cc]);
    }
#pragma unroll
    for (int q = 0; q < NT / 2; ++q) {
      const bf16x8 m0 = acc_pair(M[2 * q][0], M[2 * q + 1][0]);
      const bf16x8 m1 = acc_pair(M[2 * q][1], M[2 * q + 1][1]);
#pragma unroll
      for (int bi = 0; bi < 2; ++bi) {
        dl[bi][0] = mma_k32(dl[bi][0], wf[q][bi], m0);
        dl[bi][1] = mma_k32(dl[bi][1], wf[q][bi], m1);
      }
    }
    // scale the rows by 2^{G_31 - G_i}; decay the state; M += K^T Delta
    bf16x8 dfr[2];
#pragma unroll
    for (int cc = 0; cc < 2; ++cc)
      dfr[cc] = as_bf16x8(make_uint4(pack_bf16x2(dl[0][cc][0] * e0.x, dl[0][cc][1] * e0.y),
                                     pack_bf16x2(dl[0][cc][2] * e0.z, dl[0][cc][3] * e0.w),
                                     pack_bf16x2(dl[1][cc][0] * e1.x, dl[1][cc][1] * e1.y),
                                     pack_bf16x2(dl[1][cc][2] * e1.z, dl[1][cc][3] * e1.w)));
#pragma unroll
    for (int td = 0; td < NT; ++td)
#pragma unroll
      for (int cc = 0; cc < 2; ++cc) {
#pragma unroll
        for (int r = 0; r < 4; ++r) M[td][cc][r] *= decay;
        M[td][cc] = mma_k32(M[td][cc], kt[td], dfr[cc]);
      }
  };

  // ---- prologue: K(0) resident, K(1) and the state in registers
  load_rows(Kplane, 0, pk);
  store_rows(kbuf(0), pk);
  load_rows(Kplane, 1, pk);
#pragma unroll
  for (int td = 0; td < NT; ++td)
#pragma unroll
    for (int cc = 0; cc < 2; ++cc) {
      M[td][cc] = zero4();
      if (st_in) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          M[td][cc][r] = st_in[state_base + (size_t)(16 * td + 4 * g + r) * D + 32 * sw + 16 * cc + li];
      }
    }

  lds_barrier();                    // publishes K(0) to the prep waves

  // ---- steps -4 .. nsc-1: the state lines of sub-chunk n; K(n+5) and
  // V(n+1) go to their slots from registers loaded a step earlier
  // (the staging goes first so its LDS writes and loads overlap the step)
  for (int n = -4; n < nsc; ++n) {
    if (n + 5 < nsc) store_rows(kbuf(n + 5), pk);
    load_rows(Kplane, n + 6, pk);
    if (n + 1 >= 0 && n + 1 < nsc) store_rows(vbuf(n + 1), pv);
    load_rows(Vplane, n + 2, pv);
    if (n >= 0) state_step(n);
    lds_barrier();
  }

  float* out = st_out + state_base;
#pragma unroll
  for (int td = 0; td < NT; ++td)
#pragma unroll
    for (int cc = 0; cc < 2; ++cc)
#pragma unroll
      for (int r = 0; r < 4; ++r) out[(size_t)(16 * td + 4 * g + r) * D + 32 * sw + 16 * cc + li] = M[td][cc][r];
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
