// Chunked Gated DeltaNet state accumulation for suffix replay: the fp32
// operand path (v_mfma_f32_32x32x2f32); bf16 operands use gdn_scan_bf16.hip.
//
// Evaluates, for each (layer, segment, value head), the final state of the
// recurrence S_t = alpha_t S_{t-1}(I - beta_t k_t k_t^T) + beta_t v_t k_t^T
// (Section 2.1, Eq. recurrence) over the segment's rows, starting from zero
// (Section 1, Eq. 2) or from a given state, and stores M = S^T.  No queries or
// outputs are formed: replay only needs the state (Section 5.2).
//
// Chunked form (unrolling Eq. recurrence over a chunk of C = 64 rows that
// starts from M0, with G_i the in-chunk prefix sum of g = log alpha):
//   A_ij  = beta_i e^{G_i - G_j} k_i.k_j  (i > j)        T = (I + A)^{-1}
//   U     = T diag(beta) V                              W = T diag(beta e^G) K
//   Delta = U - W M0
//   M_C   = e^{G_C} M0 + K^T diag(e^{G_C - G}) Delta
// Only differences G_i - G_j <= 0 are exponentiated, so strong decay
// underflows to zero instead of overflowing.
//
// One workgroup per unit of max(d/32, 4) waves.  State wave w (w < d/32) owns
// state columns [32w, 32w+32) as d/32 MFMA accumulator tiles that stay in
// registers for the whole segment; at d < 128 the other waves take the Gram
// tiles and W = Tw K, so the state waves' chain of products is shorter.
// Operand precision: K and V arrive rounded once (bf16); beta and the decay
// factors are folded into T (rounded once) and into Delta (rounded once), so no
// value is rounded twice.  The state is fp32 throughout.  The two products
// that touch the state (W M0 and K^T Delta') take the state / Delta operand
// straight from accumulator registers: the MFMA k index is permuted to match
// the accumulator row layout and the other operand is read with the same
// permutation.
//
// T is built blockwise: the four 16x16 diagonal blocks by forward
// substitution (one lane per column), then block rows 1..3 with fp32 MFMA:
// T_bc = -T_bb * sum_{m=c}^{b-1} A_bm T_mc.
#include "sr_device.hpp"

#include <cstddef>
#include <type_traits>

namespace sr {
namespace {

constexpr int kC = 64;       // chunk rows
constexpr int kFP = 68;      // fp32 pitch of A and T
constexpr float kLog2e = 1.4426950408889634f;

template <typename OP, int D>
struct ScanCfg {
  static constexpr int NSW = D / 32;                   // state waves: wave w owns columns [32w, 32w+32)
  static constexpr int NW = NSW < 4 ? 4 : NSW;          // waves: the rest share the chunk products
  static constexpr int THREADS = 64 * NW;
  static constexpr int EB = std::is_same<OP, float>::value ? 4 : 2;
  static constexpr int PADE = 16 / EB;
  static constexpr int KP = D + PADE;      // pitch of Kr and W (elements)
  static constexpr int CP = kC + PADE;     // pitch of Kt, Vt, Tu, Tw
  static constexpr int R1_KR = kC * KP * EB;
  static constexpr int R1_A = kC * kFP * 4;
  static constexpr int R1_T2 = 2 * kC * CP * EB;
  static constexpr int R1 = R1_KR > R1_A ? (R1_KR > R1_T2 ? R1_KR : R1_T2) : (R1_A > R1_T2 ? R1_A : R1_T2);
  static constexpr int R2 = D * CP * EB;   // Kt
  static constexpr int R3 = D * CP * EB;   // Vt
  static constexpr int R4 = kC * kFP * 4;  // T
  static constexpr int OFF_R2 = R1, OFF_R3 = R1 + R2, OFF_R4 = R1 + R2 + R3;
  static constexpr int OFF_VEC = OFF_R4 + R4;           // 5 x 64 floats
  static constexpr int LDS = OFF_VEC + 5 * kC * 4;
  static constexpr int PIECES = kC * D * EB / 16;       // 16-byte pieces of a chunk
  static constexpr int PER_T = PIECES / THREADS;        // per thread
  static constexpr int VPP = 16 / EB;                   // elements per piece
  static constexpr int PPR = D / VPP;                   // pieces per row
  static_assert(PIECES % THREADS == 0, "chunk split");
};

__device__ __forceinline__ bf16x8 pack8(const float* v) {
  uint4 u;
  u.x = f32_to_bf16_bits(v[0]) | ((uint32_t)f32_to_bf16_bits(v[1]) << 16);
  u.y = f32_to_bf16_bits(v[2]) | ((uint32_t)f32_to_bf16_bits(v[3]) << 16);
  u.z = f32_to_bf16_bits(v[4]) | ((uint32_t)f32_to_bf16_bits(v[5]) << 16);
  u.w = f32_to_bf16_bits(v[6]) | ((uint32_t)f32_to_bf16_bits(v[7]) << 16);
  return as_bf16x8(u);
}

// Standard-order operand fragment from a row-major LDS matrix.
template <typename OP>
__device__ __forceinline__ typename Mfma<OP>::frag frag_std(const char* base, int pitch, int row, int k);
template <>
__device__ __forceinline__ bf16x8 frag_std<bf16_t>(const char* base, int pitch, int row, int k) {
  return as_bf16x8(*reinterpret_cast<const uint4*>(base + ((size_t)row * pitch + k) * 2));
}
template <>
__device__ __forceinline__ float frag_std<float>(const char* base, int pitch, int row, int k) {
  return *reinterpret_cast<const float*>(base + ((size_t)row * pitch + k) * 4);
}

// Operand fragment whose k slots follow the accumulator row layout of a
// 32-row tile starting at column `col0`: step s, lane half h.
template <typename OP>
__device__ __forceinline__ typename Mfma<OP>::frag frag_perm(const char* base, int pitch, int row, int col0,
                                                              int s, int h, bool negate);
template <>
__device__ __forceinline__ bf16x8 frag_perm<bf16_t>(const char* base, int pitch, int row, int col0, int s,
                                                     int h, bool negate) {
  const char* p = base + ((size_t)row * pitch + col0 + 16 * s + 4 * h) * 2;
  const uint2 lo = *reinterpret_cast<const uint2*>(p);
  const uint2 hi = *reinterpret_cast<const uint2*>(p + 16);
  uint4 u = make_uint4(lo.x, lo.y, hi.x, hi.y);
  if (negate) { u.x ^= 0x80008000u; u.y ^= 0x80008000u; u.z ^= 0x80008000u; u.w ^= 0x80008000u; }
  return as_bf16x8(u);
}
template <>
__device__ __forceinline__ float frag_perm<float>(const char* base, int pitch, int row, int col0, int s, int h,
                                                  bool negate) {
  const float v = *reinterpret_cast<const float*>(base + ((size_t)row * pitch + col0 + 8 * (s >> 2) + 4 * h + (s & 3)) * 4);
  return negate ? -v : v;
}

// Accumulator registers of one 32x32 tile as the B operand of MFMA step s.
template <typename OP>
__device__ __forceinline__ typename Mfma<OP>::frag frag_acc(const f32x16& acc, int s);
template <>
__device__ __forceinline__ bf16x8 frag_acc<bf16_t>(const f32x16& acc, int s) {
  float v[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) v[q] = acc[8 * s + q];
  return pack8(v);
}
template <>
__device__ __forceinline__ float frag_acc<float>(const f32x16& acc, int s) { return acc[s]; }

template <typename OP>
__device__ __forceinline__ void store_op(char* base, int idx, float v);
template <>
__device__ __forceinline__ void store_op<bf16_t>(char* base, int idx, float v) {
  reinterpret_cast<uint16_t*>(base)[idx] = f32_to_bf16_bits(v);
}
template <>
__device__ __forceinline__ void store_op<float>(char* base, int idx, float v) {
  reinterpret_cast<float*>(base)[idx] = v;
}

// Four consecutive operand values (8- or 16-byte aligned destination).
template <typename OP>
__device__ __forceinline__ void store4_op(char* base, int idx, const float* v);
template <>
__device__ __forceinline__ void store4_op<bf16_t>(char* base, int idx, const float* v) {
  uint2 u;
  u.x = f32_to_bf16_bits(v[0]) | ((uint32_t)f32_to_bf16_bits(v[1]) << 16);
  u.y = f32_to_bf16_bits(v[2]) | ((uint32_t)f32_to_bf16_bits(v[3]) << 16);
  *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(base) + idx) = u;
}
template <>
__device__ __forceinline__ void store4_op<float>(char* base, int idx, const float* v) {
  *reinterpret_cast<float4*>(reinterpret_cast<float*>(base) + idx) = make_float4(v[0], v[1], v[2], v[3]);
}

// Scatter a 16-byte piece (VPP elements of one row) into a transposed matrix.
template <typename OP>
__device__ __forceinline__ void store_transposed(char* base, int pitch, int col, int row, const uint4& v);
template <>
__device__ __forceinline__ void store_transposed<bf16_t>(char* base, int pitch, int col, int row, const uint4& v) {
  uint16_t* p = reinterpret_cast<uint16_t*>(base);
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    p[(col + 2 * e) * pitch + row] = (uint16_t)(w[e] & 0xffffu);
    p[(col + 2 * e + 1) * pitch + row] = (uint16_t)(w[e] >> 16);
  }
}
template <>
__device__ __forceinline__ void store_transposed<float>(char* base, int pitch, int col, int row, const uint4& v) {
  float* p = reinterpret_cast<float*>(base);
  p[(col + 0) * pitch + row] = __uint_as_float(v.x);
  p[(col + 1) * pitch + row] = __uint_as_float(v.y);
  p[(col + 2) * pitch + row] = __uint_as_float(v.z);
  p[(col + 3) * pitch + row] = __uint_as_float(v.w);
}

template <typename OP, int D>
__global__ __launch_bounds__(64 * (D / 32 < 4 ? 4 : D / 32)) void gdn_scan_kernel(ScanArgs a) {
  if (a.err && *a.err) return;   // the call's table check failed: write nothing
  using CF = ScanCfg<OP, D>;
  using MF = Mfma<OP>;
  constexpr int NW = CF::NW, NSW = CF::NSW, EB = CF::EB, KP = CF::KP, CP = CF::CP;
  constexpr int NT = D / 32;  // 32-row tiles along d
  __shared__ __attribute__((aligned(16))) char smem[CF::LDS];
  __shared__ int sel;

  char* R1 = smem;
  char* Kt = smem + CF::OFF_R2;
  char* Vt = smem + CF::OFF_R3;
  float* Tm = reinterpret_cast<float*>(smem + CF::OFF_R4);
  float* gs = reinterpret_cast<float*>(smem + CF::OFF_VEC);   // raw log alpha
  float* bs = gs + kC;                                        // beta
  float* Gc = bs + kC;                                        // in-chunk prefix of g
  float* eG = Gc + kC;                                        // exp(G_i)
  float* eD = eG + kC;                                        // exp(G_C - G_i)
  float* Am = reinterpret_cast<float*>(R1);                   // A (R1 phase 2)
  char* Tu = R1;                                              // R1 phase 3
  char* Tw = R1 + kC * CP * EB;
  char* Wr = R1;                                              // R1 phase 4

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int fr = lane & 31, h2 = lane >> 5;
  const int fk = h2 * MF::HALF;
  const bool state_wave = NSW == NW || wid < NSW;   // compile-time true when every wave holds state

  const int u = blockIdx.x;
  const int head = u % a.H_v;
  const int layer = (u / a.H_v) % a.n_layers;
  const int rank = u / (a.H_v * a.n_layers);
  const int b = segment_of_rank(a, rank, &sel);
  const int slot = a.slot_ids ? a.slot_ids[b] : b;
  if (slot < 0) return;
  const int64_t s0 = a.cu[b], s1 = a.cu[b + 1];
  const int hk = (head * a.H_k) / a.H_v;

  const char* Kplane = static_cast<const char*>(a.Kbuf) + (layer * a.k_layer_stride + (int64_t)hk * a.T * D) * EB;
  const char* Vplane = static_cast<const char*>(a.Vbuf) + (layer * a.v_layer_stride + (int64_t)head * a.T * D) * EB;
  const float* Gp = a.Gbuf + layer * a.g_layer_stride + (int64_t)head * a.T;
  const float* Bp = a.Bbuf + layer * a.g_layer_stride + (int64_t)head * a.T;
  // Per-layer state pointers: read from the kernel-argument segment at a
  // uniform offset (ScanArgs is the kernel's only argument, at offset 0), so
  // the 2 x kScanMaxLayers pointers are never all held in registers.
  const char* kargs = (const char*)__builtin_amdgcn_kernarg_segment_ptr();
  const float* st_in = *reinterpret_cast<const float* const*>(kargs + offsetof(ScanArgs, state_in) + sizeof(void*) * layer);
  float* st_out = *reinterpret_cast<float* const*>(kargs + offsetof(ScanArgs, state_out) + sizeof(void*) * layer);

  // T's strictly upper 16x16 blocks stay zero for the whole segment.
  for (int i = tid; i < kC * kFP; i += CF::THREADS) Tm[i] = 0.f;

  // State tiles (state waves): M[td] covers rows [32 td, 32 td + 32),
  // columns [32 wid, +32).
  f32x16 M[NT];
  const size_t state_base = ((size_t)slot * a.H_v + head) * D * D;
#pragma unroll
  for (int td = 0; td < NT; ++td) {
    if (st_in && state_wave) {
#pragma unroll
      for (int r = 0; r < 16; ++r)
        M[td][r] = st_in[state_base + (size_t)(32 * td + acc_row(r, lane)) * D + 32 * wid + fr];
    } else {
      M[td] = zero16();
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
        pk[i] = *reinterpret_cast<const uint4*>(Kplane + (t * D + cc * CF::VPP) * EB);
        pv[i] = *reinterpret_cast<const uint4*>(Vplane + (t * D + cc * CF::VPP) * EB);
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
  __syncthreads();

  for (int64_t c0 = s0; c0 < s1; c0 += kC) {
    // ---- 1. stage the chunk: K row-major (R1) and transposed, V transposed
#pragma unroll
    for (int i = 0; i < CF::PER_T; ++i) {
      const int p = tid + i * CF::THREADS;
      const int row = p / CF::PPR, cc = p % CF::PPR;
      *reinterpret_cast<uint4*>(R1 + (row * KP + cc * CF::VPP) * EB) = pk[i];
      store_transposed<OP>(Kt, CP, cc * CF::VPP, row, pk[i]);
      store_transposed<OP>(Vt, CP, cc * CF::VPP, row, pv[i]);
    }
    if (tid < kC) {
      gs[tid] = pg * kLog2e;   // log2 alpha: every decay factor below is an exp2
      bs[tid] = pb;
    }
    lds_barrier();
    if (c0 + kC < s1) prefetch(c0 + kC);

    // ---- 2. in-chunk prefix of log alpha (wave 0); Gram tiles K K^T
    if (wid == 0) {
      float x = gs[lane];
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const float y = __shfl_up(x, off);
        if (lane >= off) x += y;
      }
      const float gC = __shfl(x, 63);
      Gc[lane] = x;
      eG[lane] = exp2f(x);
      eD[lane] = exp2f(gC - x);
    }
    // lower 32x32 tiles q = 0, 1, 2 -> (0,0), (1,0), (1,1); wave w owns q = w + n NW
    constexpr int GT = (3 + NW - 1) / NW;
    f32x16 gam[GT];
#pragma unroll
    for (int n = 0; n < GT; ++n) {
      gam[n] = zero16();
      const int q = wid + n * NW;
      if (q >= 3) continue;
      const int ti = (q + 1) >> 1, tj = q >> 1;
#pragma unroll
      for (int s = 0; s < D / MF::K; ++s) {
        const auto fa = frag_std<OP>(R1, KP, 32 * ti + fr, s * MF::K + fk);
        const auto fb = frag_std<OP>(R1, KP, 32 * tj + fr, s * MF::K + fk);
        MF::mma(gam[n], fa, fb);
      }
    }
    lds_barrier();

    // ---- 3. A_ij = beta_i e^{G_i - G_j} Gamma_ij for i > j (fp32, into R1)
#pragma unroll
    for (int n = 0; n < GT; ++n) {
      const int q = wid + n * NW;
      if (q >= 3) continue;
      const int ti = (q + 1) >> 1, tj = q >> 1;
      const int j = 32 * tj + fr;
      const float gj = Gc[j];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = 32 * ti + acc_row(r, lane);
        Am[i * kFP + j] = (i > j) ? bs[i] * exp2f(fminf(Gc[i] - gj, 0.f)) * gam[n][r] : 0.f;
      }
    }
    lds_barrier();

    // ---- 4. diagonal 16x16 blocks of T = (I + A)^{-1}: lane = (block, column),
    //         column-sweep forward substitution (16-step dependency chain)
    if (wid == 0) {
      const int bb = lane >> 4, c = lane & 15;
      const float* Ab = Am + (16 * bb) * kFP + 16 * bb;
      float x[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) x[i] = (i == c) ? 1.f : 0.f;
#pragma unroll
      for (int m = 0; m < 15; ++m)
#pragma unroll
        for (int i = m + 1; i < 16; ++i) x[i] = fmaf(-Ab[i * kFP + m], x[m], x[i]);
#pragma unroll
      for (int i = 0; i < 16; ++i) Tm[(16 * bb + i) * kFP + 16 * bb + c] = x[i];
    }
    lds_barrier();

    // ---- 5. block rows 1..3: T_bc = -T_bb sum_{m=c}^{b-1} A_bm T_mc (fp32 MFMA)
    {
      const int i16 = lane & 15, k4 = lane >> 4;
#pragma unroll
      for (int lv = 1; lv < 4; ++lv) {
        for (int c = wid; c < lv; c += NW) {
          f32x4 Y = {0.f, 0.f, 0.f, 0.f};
          for (int m = c; m < lv; ++m) {
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
              const float fa = Am[(16 * lv + i16) * kFP + 16 * m + 4 * ks + k4];
              const float fb = Tm[(16 * m + 4 * ks + k4) * kFP + 16 * c + i16];
              Y = __builtin_amdgcn_mfma_f32_16x16x4f32(fa, fb, Y, 0, 0, 0);
            }
          }
          f32x4 Z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int s = 0; s < 4; ++s) {
            const float fa = Tm[(16 * lv + i16) * kFP + 16 * lv + 4 * k4 + s];
            Z = __builtin_amdgcn_mfma_f32_16x16x4f32(fa, Y[s], Z, 0, 0, 0);
          }
#pragma unroll
          for (int r = 0; r < 4; ++r) Tm[(16 * lv + 4 * k4 + r) * kFP + 16 * c + i16] = -Z[r];
        }
        lds_barrier();
      }
    }

    // ---- 6. Tu = T diag(beta), Tw = T diag(beta e^G), rounded once (into R1)
    for (int e = 4 * tid; e < kC * kC; e += 4 * CF::THREADS) {
      const int i = e >> 6, j = e & 63;
      const float4 t = *reinterpret_cast<const float4*>(Tm + i * kFP + j);
      const float4 b4 = *reinterpret_cast<const float4*>(bs + j);
      const float4 g4 = *reinterpret_cast<const float4*>(eG + j);
      const float u[4] = {t.x * b4.x, t.y * b4.y, t.z * b4.z, t.w * b4.w};
      const float v[4] = {u[0] * g4.x, u[1] * g4.y, u[2] * g4.z, u[3] * g4.w};
      store4_op<OP>(Tu, i * CP + j, u);
      store4_op<OP>(Tw, i * CP + j, v);
    }
    lds_barrier();

    // ---- 7. U = Tu V (state waves, their columns); W = Tw K, 2 NT tiles
    //         over the waves past the state waves (over all of them when
    //         every wave holds state)
    constexpr int WW0 = NW > NSW ? NSW : 0, NWW = NW - WW0;
    constexpr int WT = (2 * NT + NWW - 1) / NWW;    // W tiles per wave
    f32x16 Uacc[2], Wacc[WT];
    if (state_wave) {
#pragma unroll
      for (int ti = 0; ti < 2; ++ti) {
        Uacc[ti] = zero16();
#pragma unroll
        for (int s = 0; s < kC / MF::K; ++s) {
          const auto fa = frag_std<OP>(Tu, CP, 32 * ti + fr, s * MF::K + fk);
          const auto fb = frag_std<OP>(Vt, CP, 32 * wid + fr, s * MF::K + fk);
          MF::mma(Uacc[ti], fa, fb);
        }
      }
    }
#pragma unroll
    for (int n = 0; n < WT; ++n) {
      const int q = wid - WW0 + n * NWW;
      Wacc[n] = zero16();
      if ((WW0 > 0 && wid < WW0) || q >= 2 * NT) continue;
      const int ti = q / NT, td = q % NT;
#pragma unroll
      for (int s = 0; s < kC / MF::K; ++s) {
        const auto fa = frag_std<OP>(Tw, CP, 32 * ti + fr, s * MF::K + fk);
        const auto fb = frag_std<OP>(Kt, CP, 32 * td + fr, s * MF::K + fk);
        MF::mma(Wacc[n], fa, fb);
      }
    }
    lds_barrier();

    // ---- 8. W to R1, row-major, rounded once
#pragma unroll
    for (int n = 0; n < WT; ++n) {
      const int q = wid - WW0 + n * NWW;
      if ((WW0 > 0 && wid < WW0) || q >= 2 * NT) continue;
      const int ti = q / NT, td = q % NT;
#pragma unroll
      for (int r = 0; r < 16; ++r) store_op<OP>(Wr, (32 * ti + acc_row(r, lane)) * KP + 32 * td + fr, Wacc[n][r]);
    }
    lds_barrier();

    // ---- 9. Delta = U - W M0 (state from registers), Delta' = e^{G_C - G} Delta
    if (state_wave) {
    typename MF::frag dfrag[2][32 / MF::K];
#pragma unroll
    for (int ti = 0; ti < 2; ++ti) {
      f32x16 acc = Uacc[ti];
#pragma unroll
      for (int td = 0; td < NT; ++td) {
#pragma unroll
        for (int s = 0; s < 32 / MF::K; ++s) {
          const auto fa = frag_perm<OP>(Wr, KP, 32 * ti + fr, 32 * td, s, h2, true);
          const auto fb = frag_acc<OP>(M[td], s);
          MF::mma(acc, fa, fb);
        }
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] *= eD[32 * ti + acc_row(r, lane)];
#pragma unroll
      for (int s = 0; s < 32 / MF::K; ++s) dfrag[ti][s] = frag_acc<OP>(acc, s);
    }

    // ---- 10. M = e^{G_C} M0 + K^T Delta'
    const float eGC = eG[kC - 1];
#pragma unroll
    for (int td = 0; td < NT; ++td) {
#pragma unroll
      for (int r = 0; r < 16; ++r) M[td][r] *= eGC;
#pragma unroll
      for (int ti = 0; ti < 2; ++ti)
#pragma unroll
        for (int s = 0; s < 32 / MF::K; ++s) {
          const auto fa = frag_perm<OP>(Kt, CP, 32 * td + fr, 32 * ti, s, h2, false);
          MF::mma(M[td], fa, dfrag[ti][s]);
        }
    }
    }
    lds_barrier();
  }

  if (!state_wave) return;
  float* out = st_out + state_base;
#pragma unroll
  for (int td = 0; td < NT; ++td)
#pragma unroll
    for (int r = 0; r < 16; ++r) out[(size_t)(32 * td + acc_row(r, lane)) * D + 32 * wid + fr] = M[td][r];
}

template <typename OP, int D>
hipError_t run_scan(const ScanArgs& a, hipStream_t s) {
  const int64_t units = (int64_t)a.n_seg * a.n_layers * a.H_v;
  if (units == 0) return hipSuccess;
  hipLaunchKernelGGL((gdn_scan_kernel<OP, D>), dim3((unsigned)units), dim3(ScanCfg<OP, D>::THREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_scan(int op_dtype, int d_head, const ScanArgs& a, hipStream_t s) {
  if (op_dtype == SR_BF16) return launch_scan_bf16(d_head, a, s);
  if (op_dtype == SR_F32) {
    switch (d_head) {
      case 32: return run_scan<float, 32>(a, s);
      case 64: return run_scan<float, 64>(a, s);
      case 128: return run_scan<float, 128>(a, s);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace sr
