// Chunked Gated DeltaNet state accumulation, bf16 operands (gfx950).
//
// Same chunked form as the fp32 kernel (gdn_scan.hip), for C = 64 rows that
// start from state M0, G = in-chunk prefix of log alpha:
//   A_ij  = beta_i e^{G_i - G_j} k_i.k_j  (i > j)        T = (I + A)^{-1}
//   U     = T diag(beta) V                              W = T diag(beta e^G) K
//   Delta = U - W M0
//   M_C   = e^{G_C} M0 + K^T diag(e^{G_C - G}) Delta
//
// Layout for MI355X: d/16 waves per unit; wave w owns state columns
// [16w, 16w+16) as d/16 16x16 fp32 accumulator tiles (32 registers at d=128),
// all products are v_mfma_f32_16x16x32_bf16.  K and V stay row-major in LDS
// (plain 16-byte staging stores); every operand whose reduction index runs
// down the rows of a row-major LDS matrix (V and K for U and W, K^T for the
// state update, W for W M0) is read with ds_read_b64_tr_b16, which hands lane
// i of each 16-lane group the 4 consecutive rows kbase..kbase+3 of column
// n0 + i when lane j of the group addresses row kbase + j/4, columns
// n0 + 4 (j%4) .. +3.  The two state products take the state / Delta operand
// straight from accumulator registers, with the MFMA k slots permuted to the
// accumulator row order and the other operand read in the same order.
//
// LDS (d = 128): K, V, A (fp32), T (fp32), Tu | Tw, W^T, each ~18 KB, plus
// four 64-float vectors: 108 KB; one unit (8 waves) per CU.
#include "sr_device.hpp"

#include <cstddef>

namespace sr {
namespace {

constexpr int kC = 64;       // chunk rows
constexpr int kFP = 68;      // fp32 pitch of A
constexpr int kTP = 72;      // fp32 pitch of T
constexpr int kSortMax = 256;
constexpr float kLog2e = 1.4426950408889634f;

typedef short v4i16 __attribute__((ext_vector_type(4)));

// LDS is addressed through address-space-3 pointers with 32-bit offsets so
// that the per-read constants fold into the instructions' offset field
// instead of occupying one address register per read.
#define SR_LDS __attribute__((address_space(3)))
typedef SR_LDS char lchar;

typedef unsigned int nu32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int nu32x2 __attribute__((ext_vector_type(2)));
typedef float nf32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 lds_ld16(const lchar* p) {
  return __builtin_bit_cast(uint4, *reinterpret_cast<const SR_LDS nu32x4*>(p));
}
__device__ __forceinline__ float4 lds_ldf4(const lchar* p) {
  const nf32x4 v = *reinterpret_cast<const SR_LDS nf32x4*>(p);
  return make_float4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ uint2 lds_ld8(const lchar* p) {
  return __builtin_bit_cast(uint2, *reinterpret_cast<const SR_LDS nu32x2*>(p));
}
__device__ __forceinline__ void lds_st16(lchar* p, const uint4& v) {
  *reinterpret_cast<SR_LDS nu32x4*>(p) = __builtin_bit_cast(nu32x4, v);
}
__device__ __forceinline__ void lds_st8(lchar* p, const uint2& v) {
  *reinterpret_cast<SR_LDS nu32x2*>(p) = __builtin_bit_cast(nu32x2, v);
}

template <int D>
struct Cfg {
  static constexpr int NW = D / 16;
  static constexpr int THREADS = 64 * NW;
  static constexpr int NT = D / 16;               // 16-row tiles along d
  static constexpr int KP = D + 16;               // K / V row pitch (bf16): 4 rows hit 32 distinct banks
  static constexpr int WP = kC + 8;               // W^T, Tu, Tw row pitch (bf16)
  static constexpr int SZ_KV = kC * KP * 2;
  static constexpr int SZ_A = kC * kFP * 4;           // A, fp32
  static constexpr int SZ_T = kC * kTP * 4;           // T, fp32
  static constexpr int SZ_TUW = 2 * kC * WP * 2;      // Tu | Tw, bf16
  static constexpr int SZ_W = D * WP * 2;             // W^T, bf16
  static constexpr int OFF_K = 0, OFF_V = SZ_KV, OFF_A = 2 * SZ_KV, OFF_T = OFF_A + SZ_A;
  static constexpr int OFF_TUW = OFF_T + SZ_T, OFF_W = OFF_TUW + SZ_TUW;
  static constexpr int OFF_VEC = OFF_W + SZ_W;
  static constexpr int LDS = OFF_VEC + 4 * kC * 4;
  static constexpr int PPR = D / 8;                   // 16-byte pieces per row
  static constexpr int PER_T = kC * PPR / THREADS;    // pieces per thread (= 2)
  static constexpr int EPT = kC * kC / (4 * THREADS); // float4 of T per thread
  static_assert(kC * PPR % THREADS == 0, "staging split");
};

__device__ __forceinline__ f32x4 mma16(const f32x4& c, const bf16x8& a, const bf16x8& b) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

__device__ __forceinline__ bf16x8 ld16(const lchar* p) { return as_bf16x8(lds_ld16(p)); }

// Transposed read: with lane j of each 16-lane group pointing at row
// kbase + j/4, columns n0 + 4 (j%4) .. +3 of a row-major bf16 matrix, lane i
// receives rows kbase..kbase+3 of column n0 + i.  `p` already includes the
// lane part ((j/4) * pitch + 4 (j%4)) * 2.
__device__ __forceinline__ uint2 tr4(const lchar* p) {
  const v4i16 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((SR_LDS v4i16*)p);
  return __builtin_bit_cast(uint2, v);
}

__device__ __forceinline__ bf16x8 join(uint2 lo, uint2 hi, bool negate) {
  uint4 u = make_uint4(lo.x, lo.y, hi.x, hi.y);
  if (negate) { u.x ^= 0x80008000u; u.y ^= 0x80008000u; u.z ^= 0x80008000u; u.w ^= 0x80008000u; }
  return as_bf16x8(u);
}

__device__ __forceinline__ uint32_t pack2(float a, float b) { return pack_bf16x2(a, b); }

// Two 16x16 accumulator tiles (rows 4g..4g+3 of each) as one 16x16x32 operand.
__device__ __forceinline__ bf16x8 acc_pair(const f32x4& x, const f32x4& y) {
  return as_bf16x8(make_uint4(pack2(x[0], x[1]), pack2(x[2], x[3]), pack2(y[0], y[1]), pack2(y[2], y[3])));
}

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
  lchar* Kr = L + CF::OFF_K;                               // [64][KP] bf16
  lchar* Vr = L + CF::OFF_V;                               // [64][KP] bf16
  SR_LDS float* Am = (SR_LDS float*)(L + CF::OFF_A);       // [64][kFP] fp32
  lchar* Wt = L + CF::OFF_W;                               // [D][WP] bf16
  SR_LDS float* Tm = (SR_LDS float*)(L + CF::OFF_T);       // [64][kTP] fp32
  lchar* Tu = L + CF::OFF_TUW;                             // [64][WP] bf16
  lchar* Tw = Tu + kC * WP * 2;
  SR_LDS float* gs = (SR_LDS float*)(L + CF::OFF_VEC);     // log2 alpha
  SR_LDS float* bs = gs + kC;                              // beta
  SR_LDS float* eG = bs + kC;                              // 2^{G_i}
  SR_LDS float* eD = eG + kC;                              // 2^{G_C - G_i}

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int g = lane >> 4, li = lane & 15;
  // per-lane byte offsets; everything else is a compile-time immediate
  const int kv_row = (li * KP + 8 * g) * 2;                          // 16-byte row reads of K
  const int t_row4 = (li * WP + 4 * g) * 2;                          // 8-byte row reads of Tu / Tw
  const int tr_kv = ((li >> 2) * KP + 4 * (li & 3)) * 2;             // transposed reads of K / V
  const int tr_kv4 = tr_kv + 4 * g * KP * 2;                         //   rows 4g + ...
  const int tr_w4 = ((li >> 2) * WP + 4 * (li & 3) + 4 * g * WP) * 2; // transposed reads of W^T, rows 4g + ...

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

  // T's strictly upper 16x16 blocks stay zero for the whole segment.
  for (int i = tid; i < kC * kTP; i += CF::THREADS) Tm[i] = 0.f;

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
      const int64_t t = c0 + tid;
      pg = (t < s1) ? Gp[t] : 0.f;
      pb = (t < s1) ? Bp[t] : 0.f;
    }
  };
  if (s0 < s1) prefetch(s0);

  for (int64_t c0 = s0; c0 < s1; c0 += kC) {
    // ---- 1. stage the chunk (row-major K, V; padding rows are zero)
#pragma unroll
    for (int i = 0; i < CF::PER_T; ++i) {
      const int p = tid + i * CF::THREADS;
      const int row = p / CF::PPR, cc = p % CF::PPR;
      lds_st16(Kr + (row * KP + cc * 8) * 2, pk[i]);
      lds_st16(Vr + (row * KP + cc * 8) * 2, pv[i]);
    }
    if (tid < kC) {
      gs[tid] = pg * kLog2e;
      bs[tid] = pb;
    }
    lds_barrier();
    if (c0 + kC < s1) prefetch(c0 + kC);

    // ---- 2. in-chunk prefix G of log2 alpha (every wave, in registers);
    //         lower 16x16 tiles of K K^T;  A_ij = beta_i 2^{G_i - G_j} Gamma_ij
    float Gx = gs[lane];
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float y = __shfl_up(Gx, off);
      if (lane >= off) Gx += y;
    }
    if (wid == 0) {
      eG[lane] = exp2f(Gx);
      eD[lane] = exp2f(__shfl(Gx, 63) - Gx);
    }
    constexpr int GT = (10 + NW - 1) / NW;
#pragma unroll
    for (int n = 0; n < GT; ++n) {
      const int q = wid + n * NW;
      if (q >= 10) continue;
      const int ti = q < 1 ? 0 : q < 3 ? 1 : q < 6 ? 2 : 3;
      const int tj = q - ti * (ti + 1) / 2;
      f32x4 gam = zero4();
#pragma unroll
      for (int s = 0; s < D / 32; ++s) {
        const bf16x8 fa = ld16(Kr + kv_row + (16 * ti * KP + 32 * s) * 2);
        const bf16x8 fb = ld16(Kr + kv_row + (16 * tj * KP + 32 * s) * 2);
        gam = mma16(gam, fa, fb);
      }
      const int j = 16 * tj + li;
      const float gj = __shfl(Gx, j);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = 16 * ti + 4 * g + r;
        const float gi = __shfl(Gx, i);
        Am[i * kFP + j] = (i > j) ? bs[i] * exp2f(fminf(gi - gj, 0.f)) * gam[r] : 0.f;
      }
    }
    lds_barrier();

    // ---- 4. diagonal 16x16 blocks of T (wave 0, column-sweep substitution);
    //         the other waves clear T's strictly upper blocks
    if (wid == 0) {
      const int bb = lane >> 4, c = lane & 15;
      const SR_LDS float* Ab = Am + (16 * bb) * kFP + 16 * bb;
      float x[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) x[i] = (i == c) ? 1.f : 0.f;
      // four columns per group; the scheduling fences keep the compiler from
      // hoisting all 120 A loads at once (register pressure)
#pragma unroll
      for (int m0 = 0; m0 < 16; m0 += 4) {
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int m = m0; m < m0 + 4 && m < 15; ++m)
#pragma unroll
          for (int i = m + 1; i < 16; ++i) x[i] = fmaf(-Ab[i * kFP + m], x[m], x[i]);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < 16; ++i) Tm[(16 * bb + i) * kTP + 16 * bb + c] = x[i];
    }
    lds_barrier();

    // ---- 5. block rows 1..3: T_bc = -T_bb sum_{m=c}^{b-1} A_bm T_mc (fp32 MFMA)
    {
      const int k4 = lane >> 4;
#pragma unroll
      for (int lv = 1; lv < 4; ++lv) {
        for (int c = wid; c < lv; c += NW) {
          f32x4 Y = zero4();
          for (int m = c; m < lv; ++m) {
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
              const float fa = Am[(16 * lv + li) * kFP + 16 * m + 4 * ks + k4];
              const float fb = Tm[(16 * m + 4 * ks + k4) * kTP + 16 * c + li];
              Y = __builtin_amdgcn_mfma_f32_16x16x4f32(fa, fb, Y, 0, 0, 0);
            }
          }
          f32x4 Z = zero4();
#pragma unroll
          for (int s = 0; s < 4; ++s) {
            const float fa = Tm[(16 * lv + li) * kTP + 16 * lv + 4 * k4 + s];
            Z = __builtin_amdgcn_mfma_f32_16x16x4f32(fa, Y[s], Z, 0, 0, 0);
          }
#pragma unroll
          for (int r = 0; r < 4; ++r) Tm[(16 * lv + 4 * k4 + r) * kTP + 16 * c + li] = -Z[r];
        }
        lds_barrier();
      }
    }

    // ---- 6. Tu = T diag(beta), Tw = T diag(beta 2^G), rounded once
    {
      float4 tv[CF::EPT];
#pragma unroll
      for (int k = 0; k < CF::EPT; ++k) {
        const int e = 4 * (tid + k * CF::THREADS);
        tv[k] = lds_ldf4((const lchar*)(Tm + (e >> 6) * kTP + (e & 63)));
      }
#pragma unroll
      for (int k = 0; k < CF::EPT; ++k) {
        const int e = 4 * (tid + k * CF::THREADS);
        const int i = e >> 6, j = e & 63;
        const float4 b4 = lds_ldf4((const lchar*)(bs + j));
        const float4 g4 = lds_ldf4((const lchar*)(eG + j));
        const float u0 = tv[k].x * b4.x, u1 = tv[k].y * b4.y, u2 = tv[k].z * b4.z, u3 = tv[k].w * b4.w;
        lds_st8(Tu + (i * WP + j) * 2, make_uint2(pack2(u0, u1), pack2(u2, u3)));
        lds_st8(Tw + (i * WP + j) * 2, make_uint2(pack2(u0 * g4.x, u1 * g4.y), pack2(u2 * g4.z, u3 * g4.w)));
      }
      lds_barrier();
    }

    // ---- 7. U (this wave's 16 columns) and 4 tiles of W = Tw K, stored as W^T
    f32x4 U[4];
#pragma unroll
    for (int ti = 0; ti < 4; ++ti) {
      U[ti] = zero4();
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        // k slots of group g: rows 32s + 4g + 0..3 and 32s + 16 + 4g + 0..3
        const bf16x8 fa = join(lds_ld8(Tu + t_row4 + (16 * ti * WP + 32 * s) * 2),
                               lds_ld8(Tu + t_row4 + (16 * ti * WP + 32 * s + 16) * 2), false);
        const bf16x8 fb = join(tr4(Vr + tr_kv4 + ((32 * s) * KP + 16 * wid) * 2),
                               tr4(Vr + tr_kv4 + ((32 * s + 16) * KP + 16 * wid) * 2), false);
        U[ti] = mma16(U[ti], fa, fb);
      }
    }
    f32x4 Wacc[4];
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const int q = wid + n * NW;   // 4 NT tiles, exactly 4 per wave
      const int ti = q / NT, td = q % NT;
      Wacc[n] = zero4();
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const bf16x8 fa = join(lds_ld8(Tw + t_row4 + (16 * ti * WP + 32 * s) * 2),
                               lds_ld8(Tw + t_row4 + (16 * ti * WP + 32 * s + 16) * 2), false);
        const bf16x8 fb = join(tr4(Kr + tr_kv4 + ((32 * s) * KP + 16 * td) * 2),
                               tr4(Kr + tr_kv4 + ((32 * s + 16) * KP + 16 * td) * 2), false);
        Wacc[n] = mma16(Wacc[n], fa, fb);
      }
      // W^T tile, rounded once (the previous chunk's readers are past the
      // end-of-chunk barrier)
      lds_st8(Wt + ((16 * td + li) * WP + 16 * ti + 4 * g) * 2,
              make_uint2(pack2(Wacc[n][0], Wacc[n][1]), pack2(Wacc[n][2], Wacc[n][3])));
    }
    lds_barrier();

    // ---- 9. Delta = U - W M0 (state from registers), Delta' = 2^{G_C - G} Delta
    bf16x8 mfrag[NT / 2];   // the state as a bf16 operand, packed once per chunk
#pragma unroll
    for (int p = 0; p < NT / 2; ++p) mfrag[p] = acc_pair(M[2 * p], M[2 * p + 1]);
    f32x4 dl[4];
#pragma unroll
    for (int ti = 0; ti < 4; ++ti) {
      f32x4 acc = U[ti];
#pragma unroll
      for (int p = 0; p < NT / 2; ++p) {
        const bf16x8 fa = join(tr4(Wt + tr_w4 + ((32 * p) * WP + 16 * ti) * 2),
                               tr4(Wt + tr_w4 + ((32 * p + 16) * WP + 16 * ti) * 2), true);
        acc = mma16(acc, fa, mfrag[p]);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[r] *= eD[16 * ti + 4 * g + r];
      dl[ti] = acc;
    }
    const bf16x8 d01 = acc_pair(dl[0], dl[1]);
    const bf16x8 d23 = acc_pair(dl[2], dl[3]);

    // ---- 10. M = 2^{G_C} M0 + K^T Delta'
    const float eGC = eG[kC - 1];
#pragma unroll
    for (int td = 0; td < NT; ++td) {
#pragma unroll
      for (int r = 0; r < 4; ++r) M[td][r] *= eGC;
      const bf16x8 f0 = join(tr4(Kr + tr_kv4 + (16 * td) * 2), tr4(Kr + tr_kv4 + (16 * KP + 16 * td) * 2), false);
      M[td] = mma16(M[td], f0, d01);
      const bf16x8 f1 = join(tr4(Kr + tr_kv4 + (32 * KP + 16 * td) * 2), tr4(Kr + tr_kv4 + (48 * KP + 16 * td) * 2), false);
      M[td] = mma16(M[td], f1, d23);
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
