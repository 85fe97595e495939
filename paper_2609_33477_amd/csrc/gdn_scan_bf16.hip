// Chunked Gated DeltaNet state accumulation, bf16 operands (gfx950).
//
// Same recurrence as the fp32 kernel (gdn_scan.hip).  Rows are staged 64 at a
// time and processed as four 16-row sub-chunks b; within a sub-chunk that
// starts from state M0 (= S^T), with G the sub-chunk prefix of log alpha:
//   A_ij  = beta_i e^{G_i - G_j} k_i.k_j  (i > j)        T = (I + A)^{-1}  (16x16)
//   U     = T diag(beta) V,    W = T diag(beta e^G) K
//   Delta = U - W M0
//   M_16  = e^{G_15} M0 + K^T diag(e^{G_15 - G}) Delta
// Everything except the last two lines is independent of the state, so for
// all four sub-chunks it runs in parallel across the workgroup; the four
// state steps then run back to back in registers with no barrier.  16-row
// sub-chunks need only the 16x16 triangular inverses (no block merges) and
// cut the state-independent work per row by 4x against 64-row chunks.
//
// Layout for MI355X: d/16 waves per unit; wave w owns state columns
// [16w, 16w+16) as d/16 16x16 fp32 accumulator tiles (32 registers at d=128).
// Products use v_mfma_f32_16x16x32_bf16 (reduction over d) and
// v_mfma_f32_16x16x16_bf16 (reduction over a sub-chunk's 16 rows).  K and V
// stay row-major in LDS; operands whose reduction index runs down the rows of
// an LDS matrix are read with ds_read_b64_tr_b16, which hands lane i of each
// 16-lane group rows kbase..kbase+3 of column n0 + i when lane j of the group
// addresses row kbase + j/4, columns n0 + 4 (j%4) .. +3.  W M0 takes the state
// straight from accumulator registers, with the MFMA k slots permuted to the
// accumulator row order and W read in the same order.
//
// LDS (d = 128): K, V, W^T (~18 KB each), A (fp32) 5 KB, Tu | Tw 5 KB,
// vectors 1 KB: 66 KB.
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
  static constexpr int NW = D / 16;                   // waves; wave w owns state columns [16w, 16w+16)
  static constexpr int THREADS = 64 * NW;
  static constexpr int NT = D / 16;                   // 16-row tiles along d
  static constexpr int KP = D + 16;                   // K / V row pitch (bf16)
  static constexpr int WP = kC + 8;                   // W^T row pitch (bf16)
  static constexpr int SZ_KV = kC * KP * 2;
  static constexpr int SZ_W = D * WP * 2;
  static constexpr int SZ_A = kC * kAP * 4;           // four 16x16 fp32 blocks
  static constexpr int SZ_T = 2 * kC * kTP * 2;       // Tu | Tw, four 16x16 bf16 blocks each
  static constexpr int OFF_K = 0, OFF_V = SZ_KV, OFF_W = 2 * SZ_KV, OFF_A = OFF_W + SZ_W;
  static constexpr int OFF_T = OFF_A + SZ_A, OFF_VEC = OFF_T + SZ_T;
  static constexpr int LDS = OFF_VEC + 4 * kC * 4;
  static constexpr int PPR = D / 8;                   // 16-byte pieces per row
  static constexpr int PER_T = kC * PPR / THREADS;    // pieces per thread
  static_assert(kC * PPR % THREADS == 0, "staging split");
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
__global__ __launch_bounds__(64 * (D / 16), 2) void gdn_scan_bf16_kernel(ScanArgs a) {
  using CF = Cfg<D>;
  constexpr int NW = CF::NW, NT = CF::NT, KP = CF::KP, WP = CF::WP;
  __shared__ __attribute__((aligned(16))) char smem[CF::LDS];
  __shared__ int sel;

  lchar* L = (lchar*)smem;
  lchar* Kr = L + CF::OFF_K;                              // [64][KP] bf16
  lchar* Vr = L + CF::OFF_V;                              // [64][KP] bf16
  lchar* Wt = L + CF::OFF_W;                              // [D][WP] bf16, W^T of the four sub-chunks
  SR_LDS float* Am = (SR_LDS float*)(L + CF::OFF_A);      // [64][kAP] fp32: block b = rows 16b..16b+15
  lchar* Tu = L + CF::OFF_T;                              // [64][kTP] bf16
  lchar* Tw = Tu + kC * kTP * 2;
  SR_LDS float* gs = (SR_LDS float*)(L + CF::OFF_VEC);    // G: log2 alpha summed from the sub-chunk start
  SR_LDS float* bs = gs + kC;                             // beta
  SR_LDS float* eG = bs + kC;                             // 2^{G_i}      (G: sub-chunk prefix, log2)
  SR_LDS float* eD = eG + kC;                             // 2^{G_15 - G_i}

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
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

  // State tile td: lane holds M[16 td + 4g + r][16 wid + li].
  f32x4 M[NT];
  const size_t state_base = ((size_t)slot * a.H_v + head) * D * D;
#pragma unroll
  for (int td = 0; td < NT; ++td) {
    M[td] = zero4();
    if (st_in) {
#pragma unroll
      for (int r = 0; r < 4; ++r) M[td][r] = st_in[state_base + (size_t)(16 * td + 4 * g + r) * D + 16 * wid + li];
    }
  }

  uint4 pk[CF::PER_T], pv[CF::PER_T];
  float pg = 0.f, pb = 0.f;
  auto prefetch = [&](int64_t c0) {
#pragma unroll
    for (int i = 0; i < CF::PER_T; ++i) {
      const int p = tid + i * CF::THREADS;
      const int row = p / CF::PPR, cc = p % CF::PPR;
      const int64_t t = c0 + row;
      if (t < s1) {
        pk[i] = *reinterpret_cast<const uint4*>(Kplane + (t * D + cc * 8) * 2);
        pv[i] = *reinterpret_cast<const uint4*>(Vplane + (t * D + cc * 8) * 2);
      } else {
        pk[i] = make_uint4(0, 0, 0, 0);
        pv[i] = make_uint4(0, 0, 0, 0);
      }
    }
    if (tid < kC) {
      // log2 alpha and beta of the row; rows past the segment end carry
      // log2 alpha = 0 and beta = 0, which makes them inert
      pg = (c0 + tid < s1) ? Gp[c0 + tid] : 0.f;
      pb = (c0 + tid < s1) ? Bp[c0 + tid] : 0.f;
    }
  };
  if (s0 < s1) prefetch(s0);

  for (int64_t c0 = s0; c0 < s1; c0 += kC) {
    // ---- 1. stage 64 rows (row-major K, V; padding rows are zero with
    //         log alpha = 0 and beta = 0, which makes them inert)
#pragma unroll
    for (int i = 0; i < CF::PER_T; ++i) {
      const int p = tid + i * CF::THREADS;
      const int row = p / CF::PPR, cc = p % CF::PPR;
      lds_st16(Kr + (row * KP + cc * 8) * 2, pk[i]);
      lds_st16(Vr + (row * KP + cc * 8) * 2, pv[i]);
    }
    if (tid < kC) {
      // wave 0: inclusive prefix of log2 alpha inside each 16-row sub-chunk
      // (one 16-lane DPP row per sub-chunk), then its last value
      float gp = pg;
      gp += dpp_row_shr<1>(gp);
      gp += dpp_row_shr<2>(gp);
      gp += dpp_row_shr<4>(gp);
      gp += dpp_row_shr<8>(gp);
      const float g15 = row_last(gp, g);
      gs[tid] = gp;
      bs[tid] = pb;
      eG[tid] = exp2f(gp);
      eD[tid] = exp2f(g15 - gp);
    }
    lds_barrier();
    if (c0 + kC < s1) prefetch(c0 + kC);

    // ---- 2. Gram blocks K_b K_b^T -> A_b = beta_i 2^{G_i - G_j} Gamma (i > j)
#pragma unroll
    for (int n = 0; n < (4 + NW - 1) / NW; ++n) {
      const int sb = wid + n * NW;   // sub-chunk
      if (sb >= 4) continue;
      f32x4 gam = zero4();
#pragma unroll
      for (int s = 0; s < D / 32; ++s)
        gam = mma_k32(gam, as_bf16x8(lds_ld16(Kr + kv_row + (16 * sb * KP + 32 * s) * 2)),
                      as_bf16x8(lds_ld16(Kr + kv_row + (16 * sb * KP + 32 * s) * 2)));
      const float gj = gs[16 * sb + li];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = 4 * g + r;
        const float gi = gs[16 * sb + i];
        Am[(16 * sb + i) * kAP + li] = (i > li) ? bs[16 * sb + i] * exp2f(fminf(gi - gj, 0.f)) * gam[r] : 0.f;
      }
    }
    lds_barrier();

    // ---- 3. T_b = (I + A_b)^{-1} by forward substitution (wave 0, lane =
    //         (sub-chunk, column)); Tu = T diag(beta), Tw = T diag(beta 2^G),
    //         rounded once, written straight from the solved columns
    if (wid == 0) {
      const int sb = g, c = li;
      const SR_LDS float* Ab = Am + 16 * sb * kAP;
      float x[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        if (i % 4 == 0) __builtin_amdgcn_sched_barrier(0);   // bound the hoisting of A loads
        float s0 = (i == c) ? 1.f : 0.f, s1 = 0.f;
#pragma unroll
        for (int q = 0; q < (i + 3) / 4; ++q) {
          const float4 v = lds_ldf4((const lchar*)(Ab + i * kAP + 4 * q));
          if (4 * q + 0 < i) s0 = fmaf(-v.x, x[4 * q + 0], s0);
          if (4 * q + 1 < i) s1 = fmaf(-v.y, x[4 * q + 1], s1);
          if (4 * q + 2 < i) s0 = fmaf(-v.z, x[4 * q + 2], s0);
          if (4 * q + 3 < i) s1 = fmaf(-v.w, x[4 * q + 3], s1);
        }
        x[i] = s0 + s1;
      }
      const float bc = bs[16 * sb + c];
      const float wc = bc * eG[16 * sb + c];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        *reinterpret_cast<SR_LDS uint16_t*>(Tu + ((16 * sb + i) * kTP + c) * 2) = f32_to_bf16_bits(x[i] * bc);
        *reinterpret_cast<SR_LDS uint16_t*>(Tw + ((16 * sb + i) * kTP + c) * 2) = f32_to_bf16_bits(x[i] * wc);
      }
    }
    lds_barrier();

    // ---- 4. U_b = Tu_b V_b (this wave's columns, kept in registers) and
    //         W_b = Tw_b K_b (4 tiles per wave, stored as W^T)
    f32x4 U[4];
#pragma unroll
    for (int sb = 0; sb < 4; ++sb)
      U[sb] = mma_k16(zero4(), as_v4(lds_ld8(Tu + t_row + 16 * sb * kTP * 2)),
                      as_v4(tr4(Vr + tr_kv + (16 * sb * KP + 16 * wid) * 2)));
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const int q = wid + n * NW;   // 4 NT tiles, exactly 4 per wave
      const int sb = q / NT, td = q % NT;
      const f32x4 w = mma_k16(zero4(), as_v4(lds_ld8(Tw + t_row + 16 * sb * kTP * 2)),
                              as_v4(tr4(Kr + tr_kv + (16 * sb * KP + 16 * td) * 2)));
      lds_st8(Wt + ((16 * td + li) * WP + 16 * sb + 4 * g) * 2,
              make_uint2(pack_bf16x2(w[0], w[1]), pack_bf16x2(w[2], w[3])));
    }
    lds_barrier();

    // ---- 5. four state steps, in registers
#pragma unroll
    for (int sb = 0; sb < 4; ++sb) {
      f32x4 dl = U[sb];
#pragma unroll
      for (int p = 0; p < NT / 2; ++p)   // Delta = U - W M0, W rows read in the state's k order
        dl = mma_k32(dl,
                     join(tr4(Wt + tr_w + ((32 * p) * WP + 16 * sb) * 2),
                          tr4(Wt + tr_w + ((32 * p + 16) * WP + 16 * sb) * 2), true),
                     acc_pair(M[2 * p], M[2 * p + 1]));
      const float4 ed = lds_ldf4((const lchar*)(eD + 16 * sb + 4 * g));
      const v4i16 dfr = as_v4(make_uint2(pack_bf16x2(dl[0] * ed.x, dl[1] * ed.y), pack_bf16x2(dl[2] * ed.z, dl[3] * ed.w)));
      const float decay = eG[16 * sb + 15];
#pragma unroll
      for (int td = 0; td < NT; ++td) {
#pragma unroll
        for (int r = 0; r < 4; ++r) M[td][r] *= decay;
        M[td] = mma_k16(M[td], as_v4(tr4(Kr + tr_kv + (16 * sb * KP + 16 * td) * 2)), dfr);
      }
    }
    lds_barrier();
  }

  float* out = st_out + state_base;
#pragma unroll
  for (int td = 0; td < NT; ++td)
#pragma unroll
    for (int r = 0; r < 4; ++r) out[(size_t)(16 * td + 4 * g + r) * D + 16 * wid + li] = M[td][r];
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
