// Chunked Gated DeltaNet with per-token outputs, for group replay chaining
// (Section 4.1: a replayed layer's output is the next layer's input).
//
// Per (segment, value head) and chunk of C = 64 rows starting from the state
// M0 (M = S^T, [d_k][d_v]), with G_i the in-chunk prefix sum of log2 alpha
// (Section 2.1, Eq. recurrence unrolled over the chunk):
//   A_ij  = beta_i 2^{G_i - G_j} k_i.k_j  (i > j)        T = (I + A)^{-1}
//   U     = T diag(beta) V,   X = K M0,   Delta = U - T diag(beta 2^G) X
//   O     = diag(2^G) Q M0 + (P o (Q K^T)) Delta,   P_ij = 2^{G_i - G_j} (i >= j)
//   M_C   = 2^{G_C} M0 + K^T diag(2^{G_C - G}) Delta
// (o_i = M_i^T q_i, the state after row i applied to its query), then the
// output gate and norm of the block: y_i = RMSNorm(o_i) * w * SiLU(z_i) per
// head, stored bf16 as row i of Y [T][H_v d].  The final M is stored like the
// state-only scan's.
//
// Every product runs on v_mfma_f32_32x32x2f32 in fp32: K, Q, V and Z arrive
// in bf16 (exact in fp32), T, Delta, X and the state never get rounded, so the
// output carries only the rounding of the block's bf16 operands.  One
// workgroup of d/32 waves per (segment, head); wave w owns columns
// [32 w, 32 w + 32) of the state, of Delta and of O.  K, Q and V rows of the
// chunk are staged in LDS (bf16, pitch d + 8); A, T and P are fp32 in LDS.
// The state-side operands come straight from accumulator registers (the k
// index of the MFMA follows the accumulator row layout, the LDS operand is
// read with the same permutation).
#include "sr_device.hpp"

#include <cstddef>

namespace sr {
namespace {

constexpr int kC = 64;         // chunk rows
constexpr int kFP = 68;        // fp32 pitch of A, T, P

template <int D>
struct OutCfg {
  static constexpr int NW = D / 32;
  static constexpr int THREADS = 64 * NW;
  static constexpr int KP = D + 8;                       // bf16 pitch of K, Q, V rows
  static constexpr int SZ_ROWS = kC * KP * 2;
  static constexpr int OFF_K = 0, OFF_Q = SZ_ROWS, OFF_V = 2 * SZ_ROWS;
  static constexpr int OFF_A = 3 * SZ_ROWS;
  static constexpr int OFF_T = OFF_A + kC * kFP * 4;
  static constexpr int OFF_P = OFF_T + kC * kFP * 4;
  static constexpr int OFF_VEC = OFF_P + kC * kFP * 4;   // gs, bs, Gc, eG, eD, bw: 6 x 64 floats
  static constexpr int OFF_SS = OFF_VEC + 6 * kC * 4;    // [NW][64] row sums of squares of O
  static constexpr int LDS = OFF_SS + NW * kC * 4;
  static constexpr int PIECES = kC * D / 8;              // 16-byte pieces of one chunk matrix
  static constexpr int PER_T = PIECES / THREADS;
  static_assert(PIECES % THREADS == 0, "chunk split");
};

__device__ __forceinline__ float lds_bf16(const char* base, int idx) {
  return __uint_as_float((uint32_t)reinterpret_cast<const uint16_t*>(base)[idx] << 16);
}
// four consecutive bf16 values (idx a multiple of 4) as fp32, one 8-byte read
__device__ __forceinline__ void lds_bf16x4(const char* base, int idx, float* v) {
  const uint2 u = *reinterpret_cast<const uint2*>(base + idx * 2);
  v[0] = __uint_as_float(u.x << 16);
  v[1] = __uint_as_float(u.x & 0xffff0000u);
  v[2] = __uint_as_float(u.y << 16);
  v[3] = __uint_as_float(u.y & 0xffff0000u);
}
// four consecutive fp32 values (idx a multiple of 4), one 16-byte read
__device__ __forceinline__ void lds_f32x4(const float* base, int idx, float* v) {
  const float4 u = *reinterpret_cast<const float4*>(base + idx);
  v[0] = u.x;
  v[1] = u.y;
  v[2] = u.z;
  v[3] = u.w;
}

__device__ __forceinline__ float silu(float x) { return x * __builtin_amdgcn_rcpf(1.f + __expf(-x)); }

__device__ __forceinline__ void mma(f32x16& c, float a, float b) {
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// k index (row of the accumulator tile) of step s for lane half h
__device__ __forceinline__ int perm_k(int s, int h) { return 8 * (s >> 2) + 4 * h + (s & 3); }

template <int D>
__global__ __launch_bounds__(64 * (D / 32)) void gdn_output_kernel(OutputArgs a) {
  if (a.err && *a.err) return;   // the call's table check failed: write nothing
  using CF = OutCfg<D>;
  constexpr int NW = CF::NW, KP = CF::KP, NT = D / 32;
  __shared__ __attribute__((aligned(16))) char smem[CF::LDS];
  __shared__ int sel;
  char* Ks = smem + CF::OFF_K;
  char* Qs = smem + CF::OFF_Q;
  char* Vs = smem + CF::OFF_V;
  float* Am = reinterpret_cast<float*>(smem + CF::OFF_A);
  float* Tm = reinterpret_cast<float*>(smem + CF::OFF_T);
  float* Pm = reinterpret_cast<float*>(smem + CF::OFF_P);
  float* gs = reinterpret_cast<float*>(smem + CF::OFF_VEC);   // log2 alpha
  float* bs = gs + kC;                                        // beta
  float* Gc = bs + kC;                                        // in-chunk prefix of log2 alpha
  float* eG = Gc + kC;                                        // 2^{G_i}
  float* eD = eG + kC;                                        // 2^{G_C - G_i}
  float* bw = eD + kC;                                        // beta_i 2^{G_i}
  float* SS = reinterpret_cast<float*>(smem + CF::OFF_SS);

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int lc = lane & 31, h2 = lane >> 5;

  const int u = blockIdx.x;
  const int head = u % a.H_v;
  const int rank = u / a.H_v;
  const int b = segment_of_rank(a, rank, &sel);
  const int slot = a.slot_ids ? a.slot_ids[b] : b;
  if (slot < 0) return;
  const int64_t s0 = a.cu[b], s1 = a.cu[b + 1];
  const int hk = (head * a.H_k) / a.H_v;
  const uint16_t* Kp = static_cast<const uint16_t*>(a.Kbuf) + (int64_t)hk * a.T * D;
  const uint16_t* Qp = static_cast<const uint16_t*>(a.Qbuf) + (int64_t)hk * a.T * D;
  const uint16_t* Vp = static_cast<const uint16_t*>(a.Vbuf) + (int64_t)head * a.T * D;
  const uint16_t* Zp = static_cast<const uint16_t*>(a.Zbuf) + (int64_t)head * a.T * D;
  const float* Gp = a.Gbuf + (int64_t)head * a.T;
  const float* Bp = a.Bbuf + (int64_t)head * a.T;
  const int col = 32 * wid + lc;                        // this lane's column of Delta, O and M
  const float nw = __uint_as_float((uint32_t) static_cast<const uint16_t*>(a.norm_w)[col] << 16);
  uint16_t* Yp = static_cast<uint16_t*>(a.Y) + (int64_t)head * D + col;
  const int64_t ldy = (int64_t)a.H_v * D;

  // T's strictly upper 16x16 blocks stay zero for the whole segment
  for (int i = tid; i < kC * kFP; i += CF::THREADS) Tm[i] = 0.f;

  f32x16 M[NT];
#pragma unroll
  for (int td = 0; td < NT; ++td) M[td] = zero16();

  for (int64_t c0 = s0; c0 < s1; c0 += kC) {
    const int n = (int)(s1 - c0 < kC ? s1 - c0 : kC);   // live rows of this chunk
    // ---- 1. stage K, Q, V rows (zero past the segment end), gates
#pragma unroll
    for (int i = 0; i < CF::PER_T; ++i) {
      const int p = tid + i * CF::THREADS;
      const int row = p / (D / 8), cc = p % (D / 8);
      uint4 kv = make_uint4(0, 0, 0, 0), qv = kv, vv = kv;
      if (row < n) {
        const int64_t off = (c0 + row) * D + cc * 8;
        kv = *reinterpret_cast<const uint4*>(Kp + off);
        qv = *reinterpret_cast<const uint4*>(Qp + off);
        vv = *reinterpret_cast<const uint4*>(Vp + off);
      }
      *reinterpret_cast<uint4*>(Ks + (row * KP + cc * 8) * 2) = kv;
      *reinterpret_cast<uint4*>(Qs + (row * KP + cc * 8) * 2) = qv;
      *reinterpret_cast<uint4*>(Vs + (row * KP + cc * 8) * 2) = vv;
    }
    if (tid < kC) {
      gs[tid] = tid < n ? Gp[c0 + tid] : 0.f;
      bs[tid] = tid < n ? Bp[c0 + tid] : 0.f;
    }
    lds_barrier();

    // ---- 2. prefix of log2 alpha (wave 0); Gram K K^T and Q K^T tiles
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
      bw[lane] = bs[lane] * exp2f(x);
    }
    // tiles q = 0..5: (0,0), (1,0), (1,1) of K K^T, then of Q K^T
    constexpr int GQ = (6 + NW - 1) / NW;
    f32x16 gam[GQ];
#pragma unroll
    for (int nq = 0; nq < GQ; ++nq) {
      gam[nq] = zero16();
      const int q = wid + nq * NW;
      if (q >= 6) continue;
      const int tq = q % 3, ti = (tq + 1) >> 1, tj = tq >> 1;
      // K and Q are exact in bf16: bf16 MFMA with fp32 accumulation
      const char* Lsrc = q < 3 ? Ks : Qs;
#pragma unroll
      for (int s = 0; s < D / 16; ++s) {
        const bf16x8 fa = as_bf16x8(*reinterpret_cast<const uint4*>(Lsrc + ((32 * ti + lc) * KP + 16 * s + 8 * h2) * 2));
        const bf16x8 fb = as_bf16x8(*reinterpret_cast<const uint4*>(Ks + ((32 * tj + lc) * KP + 16 * s + 8 * h2) * 2));
        gam[nq] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa, fb, gam[nq], 0, 0, 0);
      }
    }
    lds_barrier();

    // ---- 3. A_ij = beta_i 2^{G_i - G_j} Gamma_ij (i > j); P_ij = 2^{G_i - G_j} (QK^T)_ij (i >= j)
#pragma unroll
    for (int nq = 0; nq < GQ; ++nq) {
      const int q = wid + nq * NW;
      if (q >= 6) continue;
      const int tq = q % 3, ti = (tq + 1) >> 1, tj = tq >> 1;
      const int j = 32 * tj + lc;
      const float gj = Gc[j];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = 32 * ti + acc_row(r, lane);
        const float dec = exp2f(fminf(Gc[i] - gj, 0.f));
        if (q < 3) Am[i * kFP + j] = (i > j) ? bs[i] * dec * gam[nq][r] : 0.f;
        else Pm[i * kFP + j] = (i >= j) ? dec * gam[nq][r] : 0.f;
      }
      if (tq == 1) {   // the strictly upper tile (0,1) of P is zero
#pragma unroll
        for (int r = 0; r < 16; ++r) Pm[(acc_row(r, lane)) * kFP + 32 + lc] = 0.f;
      }
    }
    lds_barrier();

    // ---- 4. diagonal 16x16 blocks of T = (I + A)^{-1} by forward substitution
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
    // block rows 1..3: T_bc = -T_bb sum_{m=c}^{b-1} A_bm T_mc
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

    // Operands on the k side of a state product follow the accumulator row
    // order: step s takes rows perm_k(s, h) of a 32-row tile, i.e. four runs
    // of four consecutive rows, so the LDS side is read 4 values at a time.
    // ---- 5. X = K M0 (this wave's columns), from the state registers
    f32x16 X[2];
#pragma unroll
    for (int ti = 0; ti < 2; ++ti) {
      X[ti] = zero16();
#pragma unroll
      for (int td = 0; td < NT; ++td) {
        float av[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) lds_bf16x4(Ks, (32 * ti + lc) * KP + 32 * td + 8 * q + 4 * h2, av + 4 * q);
#pragma unroll
        for (int s = 0; s < 16; ++s) mma(X[ti], av[s], M[td][s]);
      }
    }
    // ---- 6. Delta = T diag(beta) V - T diag(beta 2^G) X
    f32x16 Dl[2];
#pragma unroll
    for (int ti = 0; ti < 2; ++ti) {
      Dl[ti] = zero16();
#pragma unroll
      for (int tj = 0; tj < 2; ++tj) {
        float tv[16], bv[16], wv[16], vv[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int j0 = 32 * tj + 8 * q + 4 * h2;
          lds_f32x4(Tm, (32 * ti + lc) * kFP + j0, tv + 4 * q);
          lds_f32x4(bs, j0, bv + 4 * q);
          lds_f32x4(bw, j0, wv + 4 * q);
        }
#pragma unroll
        for (int s = 0; s < 16; ++s) vv[s] = lds_bf16(Vs, (32 * tj + perm_k(s, h2)) * KP + col);
#pragma unroll
        for (int s = 0; s < 16; ++s) mma(Dl[ti], tv[s] * bv[s], vv[s]);
#pragma unroll
        for (int s = 0; s < 16; ++s) mma(Dl[ti], -tv[s] * wv[s], X[tj][s]);
      }
    }
    // ---- 7. O = diag(2^G) Q M0 + (P o QK^T) Delta
    f32x16 O[2];
#pragma unroll
    for (int ti = 0; ti < 2; ++ti) {
      O[ti] = zero16();
#pragma unroll
      for (int td = 0; td < NT; ++td) {
        float av[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) lds_bf16x4(Qs, (32 * ti + lc) * KP + 32 * td + 8 * q + 4 * h2, av + 4 * q);
#pragma unroll
        for (int s = 0; s < 16; ++s) mma(O[ti], av[s], M[td][s]);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) O[ti][r] *= eG[32 * ti + acc_row(r, lane)];
#pragma unroll
      for (int tj = 0; tj < 2; ++tj) {
        float pv[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) lds_f32x4(Pm, (32 * ti + lc) * kFP + 32 * tj + 8 * q + 4 * h2, pv + 4 * q);
#pragma unroll
        for (int s = 0; s < 16; ++s) mma(O[ti], pv[s], Dl[tj][s]);
      }
    }
    // ---- 8. gated output norm: per row, sum of squares over the head's d columns
#pragma unroll
    for (int ti = 0; ti < 2; ++ti)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float v = O[ti][r] * O[ti][r];
#pragma unroll
        for (int off = 16; off >= 1; off >>= 1) v += __shfl_xor(v, off);   // over the 32 columns
        if (lc == 0) SS[wid * kC + 32 * ti + acc_row(r, lane)] = v;
      }
    // ---- 9. M = 2^{G_C} M0 + K^T diag(2^{G_C - G}) Delta
    const float eGC = eG[kC - 1];
#pragma unroll
    for (int tj = 0; tj < 2; ++tj)
#pragma unroll
      for (int r = 0; r < 16; ++r) Dl[tj][r] *= eD[32 * tj + acc_row(r, lane)];
#pragma unroll
    for (int td = 0; td < NT; ++td) {
#pragma unroll
      for (int r = 0; r < 16; ++r) M[td][r] *= eGC;
#pragma unroll
      for (int tj = 0; tj < 2; ++tj) {
        float kv[16];
#pragma unroll
        for (int s = 0; s < 16; ++s) kv[s] = lds_bf16(Ks, (32 * tj + perm_k(s, h2)) * KP + 32 * td + lc);
#pragma unroll
        for (int s = 0; s < 16; ++s) mma(M[td], kv[s], Dl[tj][s]);
      }
    }
    lds_barrier();
    // ---- 10. y = o / sqrt(mean(o^2) + eps) * w * SiLU(z), rows of this chunk
#pragma unroll
    for (int ti = 0; ti < 2; ++ti)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = 32 * ti + acc_row(r, lane);
        if (i < n) {
          float ss = 0.f;
#pragma unroll
          for (int w = 0; w < NW; ++w) ss += SS[w * kC + i];
          const float inv = __builtin_amdgcn_rsqf(ss / (float)D + a.eps);
          const int64_t t = c0 + i;
          const float z = __uint_as_float((uint32_t)Zp[t * D + col] << 16);
          Yp[t * ldy] = f32_to_bf16_bits(O[ti][r] * inv * nw * silu(z));
        }
      }
    lds_barrier();   // the next chunk's staging overwrites K, Q, V and SS
  }

  float* out = a.state_out + ((size_t)slot * a.H_v + head) * D * D;
#pragma unroll
  for (int td = 0; td < NT; ++td)
#pragma unroll
    for (int r = 0; r < 16; ++r) out[(size_t)(32 * td + acc_row(r, lane)) * D + col] = M[td][r];
}

template <int D>
hipError_t run_output(const OutputArgs& a, hipStream_t s) {
  const int64_t units = (int64_t)a.n_seg * a.H_v;
  if (units == 0) return hipSuccess;
  hipLaunchKernelGGL((gdn_output_kernel<D>), dim3((unsigned)units), dim3(OutCfg<D>::THREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gdn_output(int d_head, const OutputArgs& a, hipStream_t s) {
  switch (d_head) {
    case 64: return run_output<64>(a, s);
    case 128: return run_output<128>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace sr
