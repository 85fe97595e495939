// Chunked Gated DeltaNet with per-token outputs, for group replay chaining
// (Section 4.1: a replayed layer's output is the next layer's input), and the
// same chunk algebra without outputs as the state-only scan of heads whose
// key and value widths differ (Appendix A: OLMo-Hybrid's d_k = 96,
// d_v = 192), where the pipelined scan's square tiling does not apply.
//
// Per (segment, value head) and chunk of C = 64 rows starting from the state
// M0 (M = S^T, [d_k][d_v]), with G_i the in-chunk prefix sum of log2 alpha
// (Section 2.1, Eq. recurrence unrolled over the chunk):
//   A_ij  = beta_i 2^{G_i - G_j} k_i.k_j  (i > j)        T = (I + A)^{-1}
//   X     = K M0,   R = V - diag(2^G) X,   Delta = T diag(beta) R
//   O     = diag(2^G) Q M0 + (P o (Q K^T)) Delta,   P_ij = 2^{G_i - G_j} (i >= j)
//   M_C   = 2^{G_C} M0 + K^T diag(2^{G_C - G}) Delta
// (Delta = U - W M0 of the WY form with U = T diag(beta) V and
// W = T diag(beta 2^G) K, taken as one product; o_i = M_i^T q_i, the state
// after row i applied to its query), then the output gate and norm of the
// block: y_i = RMSNorm(o_i) * w * SiLU(z_i) per head, stored bf16 as row i of
// Y [T][H_v d].  The final M is stored like the state-only scan's.
//
// Precision: A, T, Delta, O and the state stay fp32.  The products run on
// v_mfma_f32_32x32x16_bf16 with every fp32 operand split into a bf16 high
// part and a bf16 low part (x = hi + lo to 2^-18 |x|): an operand that is
// exact in bf16 (K, Q, V) takes two products (with hi and with lo), two fp32
// operands take three (hi.hi + hi.lo + lo.hi), so each product keeps about
// 16 significant bits and nothing is rounded to bf16 on the way; the output
// carries the rounding of the block's bf16 operands and of y itself.
//
// One workgroup of d_v/32 waves per (segment, head) (and layer, state-only);
// wave w owns columns [32 w, 32 w + 32) of the state, of Delta and of O,
// each a stack of 32 x 32 accumulator tiles.  A 16-deep k-step of a product
// whose reduction runs over accumulator rows (the chunk rows of X, R and
// Delta; the d_k rows of M) uses
// the k-slot order of the accumulator: slot 8h + j of lane half h is row
// 8 (j / 4) + 4 h + j % 4, so registers 8 s .. 8 s + 7 of a tile are k-step s
// of its B operand as they stand; the A operand is read from LDS in the same
// order (two 8-byte row reads, or two transposed reads for K^T).  K, Q, V, Z
// rows of the chunk are staged in LDS (bf16, pitch width + 8); A and T are
// fp32 in LDS, T diag(beta) and P bf16 hi | lo.  The output norm runs
// row-wise over an fp32 copy of O in LDS, one row per d_v/32 lanes, with
// coalesced 64-byte stores.
#include "sr_device.hpp"

#include <cstddef>

namespace sr {
namespace {

constexpr int kC = 64;         // chunk rows
constexpr int kFP = 68;        // fp32 pitch of A and T
constexpr int kBP = 68;        // bf16 pitch of the hi / lo parts of T diag(beta) and P

template <int DK, int DV, bool OUT>
struct OutCfg {
  static constexpr int NW = DV / 32;
  static constexpr int THREADS = 64 * NW;
  static constexpr int KP = DK + 8, VP = DV + 8;          // bf16 pitches of K | Q and V | Z rows
  static constexpr int OP = DV + 4;                       // fp32 pitch of the output rows
  static constexpr int SZ_K = kC * KP * 2, SZ_V = kC * VP * 2;
  static constexpr int OFF_K = 0, OFF_V = SZ_K;
  static constexpr int OFF_Q = OFF_V + SZ_V;              // Q and Z with outputs only
  static constexpr int OFF_Z = OFF_Q + (OUT ? SZ_K : 0);
  static constexpr int OFF_A = OFF_Z + (OUT ? SZ_V : 0);  // A (fp32); then, with T, the output rows
  static constexpr int OFF_T = OFF_A + kC * kFP * 4;       // T (fp32), then T diag(beta) hi | lo
  static constexpr int OFF_P = OFF_T + kC * kFP * 4;       // P hi | lo (outputs only)
  static constexpr int OFF_VEC = OFF_P + (OUT ? 2 * kC * kBP * 2 : 0);   // gs, bs, Gc, eG, eD
  static constexpr int OFF_NW = OFF_VEC + 5 * kC * 4;      // norm weight (fp32) [DV]
  static constexpr int LDS = OFF_NW + (OUT ? DV * 4 : 0);
  static constexpr int PER_K = kC * DK / 8 / THREADS;     // 16-byte pieces per thread of a K | Q chunk
  static constexpr int PER_V = kC * DV / 8 / THREADS;     // ... of a V | Z chunk
  static_assert(DK % 32 == 0 && DV % 32 == 0 && DK <= 128 && DV <= 256, "head widths");
  static_assert(kC * DK / 8 % THREADS == 0 && kC * DV / 8 % THREADS == 0, "chunk split");
  static_assert(!OUT || kC * OP * 4 <= 2 * kC * kFP * 4, "output rows in the place of A and T");
  static_assert(2 * kC * kBP * 2 <= kC * kFP * 4, "T diag(beta) hi | lo in the place of T");
};

typedef __attribute__((address_space(3))) char lchar;
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint2 ld8(const lchar* p) {
  return __builtin_bit_cast(uint2, *reinterpret_cast<const __attribute__((address_space(3))) u32x2*>(p));
}
__device__ __forceinline__ uint4 ld16(const lchar* p) {
  return __builtin_bit_cast(uint4, *reinterpret_cast<const __attribute__((address_space(3))) u32x4*>(p));
}
__device__ __forceinline__ float4 ldf4(const lchar* p) {
  const f32x4v v = *reinterpret_cast<const __attribute__((address_space(3))) f32x4v*>(p);
  return make_float4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ float lo_f(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float hi_f(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

// A-operand fragment of k-step [k0, k0 + 16) from a row-major bf16 row: slots
// 8h .. 8h + 3 are columns k0 + 4h .. + 3, slots 8h + 4 .. 8h + 7 columns
// k0 + 8 + 4h .. + 3
__device__ __forceinline__ bf16x8 frag_row(const lchar* row, int k0, int h) {
  const uint2 a = ld8(row + (k0 + 4 * h) * 2), b = ld8(row + (k0 + 8 + 4 * h) * 2);
  return as_bf16x8(make_uint4(a.x, a.y, b.x, b.y));
}

// Eight fp32 values (accumulator registers 8s .. 8s + 7) as a bf16 high part
// and the bf16 rounding of the remainder.
__device__ __forceinline__ void split8(const f32x16& v, int s, bf16x8& hi, bf16x8& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float x0 = v[8 * s + 2 * e], x1 = v[8 * s + 2 * e + 1];
    h[e] = pack_bf16x2(x0, x1);
    l[e] = pack_bf16x2(x0 - lo_f(h[e]), x1 - hi_f(h[e]));
  }
  hi = as_bf16x8(make_uint4(h[0], h[1], h[2], h[3]));
  lo = as_bf16x8(make_uint4(l[0], l[1], l[2], l[3]));
}

__device__ __forceinline__ f32x16 mma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float silu(float x) { return x * __builtin_amdgcn_rcpf(1.f + __expf(-x)); }

// A: OutputArgs (one layer, with outputs) or ScanArgs (state only, up to
// kScanMaxLayers layers per launch, initial states allowed).
template <int DK, int DV, bool OUT, typename A>
__global__ __launch_bounds__(64 * (DV / 32)) void gdn_chunk_kernel(A a) {
  if (a.err && *a.err) return;   // the call's table check failed: write nothing
  using CF = OutCfg<DK, DV, OUT>;
  constexpr int NW = CF::NW, KP = CF::KP, VP = CF::VP, NT = DK / 32, OP = CF::OP;
  __shared__ __attribute__((aligned(16))) char smem[CF::LDS];
  __shared__ int sel;
  lchar* L = (lchar*)smem;
  lchar* Ks = L + CF::OFF_K;
  lchar* Qs = L + CF::OFF_Q;
  lchar* Vs = L + CF::OFF_V;
  lchar* Zs = L + CF::OFF_Z;
  float* Am = reinterpret_cast<float*>(smem + CF::OFF_A);
  float* Tm = reinterpret_cast<float*>(smem + CF::OFF_T);
  lchar* Tbh = L + CF::OFF_T;                                   // T diag(beta): hi, then lo
  lchar* Tbl = Tbh + kC * kBP * 2;
  lchar* Ph = L + CF::OFF_P;                                    // P o (Q K^T): hi, then lo
  lchar* Pl = Ph + kC * kBP * 2;
  uint16_t* Ph16 = reinterpret_cast<uint16_t*>(smem + CF::OFF_P);
  uint16_t* Pl16 = Ph16 + kC * kBP;
  float* Os = reinterpret_cast<float*>(smem + CF::OFF_A);      // output rows (after A and T are done)
  float* gs = reinterpret_cast<float*>(smem + CF::OFF_VEC);    // log2 alpha
  float* bs = gs + kC;                                         // beta
  float* Gc = bs + kC;                                         // in-chunk prefix of log2 alpha
  float* eG = Gc + kC;                                         // 2^{G_i}
  float* eD = eG + kC;                                         // 2^{G_C - G_i}
  float* nws = reinterpret_cast<float*>(smem + CF::OFF_NW);    // norm weight

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int lc = lane & 31, h2 = lane >> 5;

  // unit -> (segment, layer, value head)
  const int u = blockIdx.x;
  const int head = u % a.H_v;
  int layer = 0, rank = u / a.H_v;
  if constexpr (!OUT) {
    layer = rank % a.n_layers;
    rank /= a.n_layers;
  }
  const int b = segment_of_rank(a, rank, &sel);
  const int slot = a.slot_ids ? a.slot_ids[b] : b;
  if (slot < 0) return;
  const int64_t s0 = a.cu[b], s1 = a.cu[b + 1];
  const int hk = (head * a.H_k) / a.H_v;
  const uint16_t* Kp;
  const uint16_t* Vp;
  int kpitch = DK;                                      // elements per K row
  const uint16_t* Qp = nullptr;
  const uint16_t* Zp = nullptr;
  const float* Gp;
  const float* Bp;
  const float* st_in = nullptr;
  float* st_out;
  if constexpr (OUT) {
    Kp = static_cast<const uint16_t*>(a.Kbuf) + (int64_t)hk * a.T * DK;
    Qp = static_cast<const uint16_t*>(a.Qbuf) + (int64_t)hk * a.T * DK;
    Vp = static_cast<const uint16_t*>(a.Vbuf) + (int64_t)head * a.T * DV;
    Zp = static_cast<const uint16_t*>(a.Zbuf) + (int64_t)head * a.T * DV;
    Gp = a.Gbuf + (int64_t)head * a.T;
    Bp = a.Bbuf + (int64_t)head * a.T;
    st_out = a.state_out;
  } else {
    if (a.k_pitch > 0) kpitch = a.k_pitch;
    Kp = static_cast<const uint16_t*>(a.Kbuf) + layer * a.k_layer_stride + (int64_t)hk * a.T * kpitch;
    Vp = static_cast<const uint16_t*>(a.Vbuf) + layer * a.v_layer_stride + (int64_t)head * a.T * DV;
    Gp = a.Gbuf + layer * a.g_layer_stride + (int64_t)head * a.T;
    Bp = a.Bbuf + layer * a.g_layer_stride + (int64_t)head * a.T;
    // per-layer state pointers from the kernel arguments at a uniform offset
    // (the argument block is the only kernel argument)
    const char* kargs = (const char*)__builtin_amdgcn_kernarg_segment_ptr();
    st_in = *reinterpret_cast<const float* const*>(kargs + offsetof(ScanArgs, state_in) + sizeof(void*) * layer);
    st_out = *reinterpret_cast<float* const*>(kargs + offsetof(ScanArgs, state_out) + sizeof(void*) * layer);
  }
  const size_t state_base = ((size_t)slot * a.H_v + head) * DK * DV;
  const int col = 32 * wid + lc;                        // this lane's column of Delta, O and M
  if constexpr (OUT) {
    if (tid < DV) nws[tid] = __uint_as_float((uint32_t) static_cast<const uint16_t*>(a.norm_w)[tid] << 16);
  }

  // transposed reads of a row-major bf16 matrix of pitch `pitch`: lane
  // (lc, h2) receives rows row0 + 4 h2 .. + 3 of column c0 + lc
  const int tr_r = lane & 15;                           // lane within its 16-lane group
  const int tr_n = 16 * ((lane >> 4) & 1) + 4 * (tr_r & 3);
  auto tr4 = [&](const lchar* base, int pitch, int row0, int c0) {
    return lds_tr4(base + ((row0 + 4 * h2 + (tr_r >> 2)) * pitch + c0 + tr_n) * 2);
  };

  f32x16 M[NT];
#pragma unroll
  for (int td = 0; td < NT; ++td) {
    M[td] = zero16();
    if (st_in) {
#pragma unroll
      for (int r = 0; r < 16; ++r) M[td][r] = st_in[state_base + (size_t)(32 * td + acc_row(r, lane)) * DV + col];
    }
  }

  for (int64_t c0 = s0; c0 < s1; c0 += kC) {
    const int n = (int)(s1 - c0 < kC ? s1 - c0 : kC);   // live rows of this chunk
    // ---- 1. stage K (, Q), V (, Z) rows (zero past the segment end), gates
    if constexpr (DK == DV) {
#pragma unroll
      for (int i = 0; i < CF::PER_K; ++i) {
        const int p = tid + i * CF::THREADS;
        const int row = p / (DK / 8), cc = p % (DK / 8);
        uint4 kv = make_uint4(0, 0, 0, 0), qv = kv, vv = kv, zv = kv;
        if (row < n) {
          const int64_t off = (c0 + row) * DK + cc * 8;
          kv = *reinterpret_cast<const uint4*>(Kp + off);
          vv = *reinterpret_cast<const uint4*>(Vp + off);
          if constexpr (OUT) {
            qv = *reinterpret_cast<const uint4*>(Qp + off);
            zv = *reinterpret_cast<const uint4*>(Zp + off);
          }
        }
        const int lo = (row * KP + cc * 8) * 2;
        *reinterpret_cast<uint4*>(smem + CF::OFF_K + lo) = kv;
        *reinterpret_cast<uint4*>(smem + CF::OFF_V + lo) = vv;
        if constexpr (OUT) {
          *reinterpret_cast<uint4*>(smem + CF::OFF_Q + lo) = qv;
          *reinterpret_cast<uint4*>(smem + CF::OFF_Z + lo) = zv;
        }
      }
    } else {
#pragma unroll
    for (int i = 0; i < CF::PER_K; ++i) {
      const int p = tid + i * CF::THREADS;
      const int row = p / (DK / 8), cc = p % (DK / 8);
      uint4 kv = make_uint4(0, 0, 0, 0), qv = kv;
      if (row < n) {
        kv = *reinterpret_cast<const uint4*>(Kp + (c0 + row) * kpitch + cc * 8);
        if constexpr (OUT) qv = *reinterpret_cast<const uint4*>(Qp + (c0 + row) * DK + cc * 8);
      }
      const int lo = (row * KP + cc * 8) * 2;
      *reinterpret_cast<uint4*>(smem + CF::OFF_K + lo) = kv;
      if constexpr (OUT) *reinterpret_cast<uint4*>(smem + CF::OFF_Q + lo) = qv;
    }
#pragma unroll
    for (int i = 0; i < CF::PER_V; ++i) {
      const int p = tid + i * CF::THREADS;
      const int row = p / (DV / 8), cc = p % (DV / 8);
      uint4 vv = make_uint4(0, 0, 0, 0), zv = vv;
      if (row < n) {
        const int64_t off = (c0 + row) * DV + cc * 8;
        vv = *reinterpret_cast<const uint4*>(Vp + off);
        if constexpr (OUT) zv = *reinterpret_cast<const uint4*>(Zp + off);
      }
      const int lo = (row * VP + cc * 8) * 2;
      *reinterpret_cast<uint4*>(smem + CF::OFF_V + lo) = vv;
      if constexpr (OUT) *reinterpret_cast<uint4*>(smem + CF::OFF_Z + lo) = zv;
    }
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
    }
    // tiles q = 0..5: (0,0), (1,0), (1,1) of K K^T, then (outputs only) of Q K^T
    constexpr int NQ = OUT ? 6 : 3;
    constexpr int GQ = (NQ + NW - 1) / NW;
    f32x16 gam[GQ];
#pragma unroll
    for (int nq = 0; nq < GQ; ++nq) {
      gam[nq] = zero16();
      const int q = wid + nq * NW;
      if (q >= NQ) continue;
      const int tq = q % 3, ti = (tq + 1) >> 1, tj = tq >> 1;
      const lchar* Lsrc = q < 3 ? Ks : Qs;
#pragma unroll
      for (int s = 0; s < DK / 16; ++s) {
        const bf16x8 fa = as_bf16x8(ld16(Lsrc + ((32 * ti + lc) * KP + 16 * s + 8 * h2) * 2));
        const bf16x8 fb = as_bf16x8(ld16(Ks + ((32 * tj + lc) * KP + 16 * s + 8 * h2) * 2));
        gam[nq] = mma(fa, fb, gam[nq]);
      }
    }
    lds_barrier();

    // ---- 3. A_ij = beta_i 2^{G_i - G_j} Gamma_ij (i > j), fp32;
    //         P_ij = 2^{G_i - G_j} (Q K^T)_ij (i >= j), bf16 hi | lo
#pragma unroll
    for (int nq = 0; nq < GQ; ++nq) {
      const int q = wid + nq * NW;
      if (q >= NQ) continue;
      const int tq = q % 3, ti = (tq + 1) >> 1, tj = tq >> 1;
      const int j = 32 * tj + lc;
      const float gj = Gc[j];
      // this lane's rows 32 ti + 8 r4 + 4 h2 .. + 3 (r4 = 0..3)
      float gi[16], bi[16];
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int i0 = 32 * ti + 8 * r4 + 4 * h2;
        const float4 g4 = ldf4((const lchar*)(Gc + i0));
        const float4 b4 = ldf4((const lchar*)(bs + i0));
        gi[4 * r4] = g4.x; gi[4 * r4 + 1] = g4.y; gi[4 * r4 + 2] = g4.z; gi[4 * r4 + 3] = g4.w;
        bi[4 * r4] = b4.x; bi[4 * r4 + 1] = b4.y; bi[4 * r4 + 2] = b4.z; bi[4 * r4 + 3] = b4.w;
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = 32 * ti + acc_row(r, lane);
        const float dec = exp2f(fminf(gi[r] - gj, 0.f));
        if (q < 3) {
          Am[i * kFP + j] = (i > j) ? bi[r] * dec * gam[nq][r] : 0.f;
        } else {
          const float v = (i >= j) ? dec * gam[nq][r] : 0.f;
          const uint32_t hv = pack_bf16x2(v, 0.f);
          Ph16[i * kBP + j] = (uint16_t)hv;
          Pl16[i * kBP + j] = (uint16_t)pack_bf16x2(v - lo_f(hv), 0.f);
        }
      }
      if (q == 4) {   // the strictly upper tile (0,1) of P is zero
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          Ph16[acc_row(r, lane) * kBP + 32 + lc] = 0;
          Pl16[acc_row(r, lane) * kBP + 32 + lc] = 0;
        }
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
    // T diag(beta) as bf16 hi | lo in T's place (the strictly upper 16x16
    // blocks of T are zero; their storage is not written for T)
    {
      constexpr int PER = (kC * kC / 4 + CF::THREADS - 1) / CF::THREADS;   // 4-column pieces per thread
      float tv[PER][4];
#pragma unroll
      for (int e = 0; e < PER; ++e) {
        const int p = tid + e * CF::THREADS, c4 = p % 16;
        const int row = (kC * kC / 4) % CF::THREADS == 0 ? p / 16 : (p / 16) & (kC - 1);   // wraps past the end: unused
        const float4 t4 = ldf4((const lchar*)(Tm + row * kFP + 4 * c4));
        const float4 b4 = ldf4((const lchar*)(bs + 4 * c4));
        const bool upper = (c4 >> 2) > (row >> 4);
        tv[e][0] = upper ? 0.f : t4.x * b4.x;
        tv[e][1] = upper ? 0.f : t4.y * b4.y;
        tv[e][2] = upper ? 0.f : t4.z * b4.z;
        tv[e][3] = upper ? 0.f : t4.w * b4.w;
      }
      lds_barrier();
#pragma unroll
      for (int e = 0; e < PER; ++e) {
        const int p = tid + e * CF::THREADS, row = p / 16, c4 = p % 16;
        if ((kC * kC / 4) % CF::THREADS != 0 && p >= kC * kC / 4) break;
        const uint32_t h0 = pack_bf16x2(tv[e][0], tv[e][1]), h1 = pack_bf16x2(tv[e][2], tv[e][3]);
        const uint32_t l0 = pack_bf16x2(tv[e][0] - lo_f(h0), tv[e][1] - hi_f(h0));
        const uint32_t l1 = pack_bf16x2(tv[e][2] - lo_f(h1), tv[e][3] - hi_f(h1));
        *reinterpret_cast<uint2*>(smem + CF::OFF_T + (row * kBP + 4 * c4) * 2) = make_uint2(h0, h1);
        *reinterpret_cast<uint2*>(smem + CF::OFF_T + kC * kBP * 2 + (row * kBP + 4 * c4) * 2) = make_uint2(l0, l1);
      }
      lds_barrier();
    }

    // ---- 5. X = K M0 and Q M0 (this wave's columns): K and Q exact in bf16,
    // M0 as hi + lo
    f32x16 X[2], O[2];
#pragma unroll
    for (int ti = 0; ti < 2; ++ti) {
      X[ti] = zero16();
      O[ti] = zero16();
    }
#pragma unroll
    for (int td = 0; td < NT; ++td) {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        bf16x8 mh, ml;
        split8(M[td], s, mh, ml);
#pragma unroll
        for (int ti = 0; ti < 2; ++ti) {
          const int off = (32 * ti + lc) * KP * 2;
          const bf16x8 ka = frag_row(Ks + off, 32 * td + 16 * s, h2);
          if constexpr (OUT) {
            const bf16x8 qa = frag_row(Qs + off, 32 * td + 16 * s, h2);
            X[ti] = mma(ka, ml, mma(ka, mh, X[ti]));
            O[ti] = mma(qa, ml, mma(qa, mh, O[ti]));
          } else {
            X[ti] = mma(ka, ml, mma(ka, mh, X[ti]));
          }
        }
      }
    }
    // ---- 6. R = V - diag(2^G) X (in X's registers); Delta = T diag(beta) R
#pragma unroll
    for (int tj = 0; tj < 2; ++tj) {
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const uint2 v4 = tr4(Vs, VP, 32 * tj + 8 * r4, 32 * wid);
        const float4 g4 = ldf4((const lchar*)(eG + 32 * tj + 8 * r4 + 4 * h2));
        X[tj][4 * r4 + 0] = fmaf(-g4.x, X[tj][4 * r4 + 0], lo_f(v4.x));
        X[tj][4 * r4 + 1] = fmaf(-g4.y, X[tj][4 * r4 + 1], hi_f(v4.x));
        X[tj][4 * r4 + 2] = fmaf(-g4.z, X[tj][4 * r4 + 2], lo_f(v4.y));
        X[tj][4 * r4 + 3] = fmaf(-g4.w, X[tj][4 * r4 + 3], hi_f(v4.y));
      }
    }
    f32x16 Dl[2];
#pragma unroll
    for (int ti = 0; ti < 2; ++ti) Dl[ti] = zero16();
#pragma unroll
    for (int tj = 0; tj < 2; ++tj)
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        bf16x8 rh, rl;
        split8(X[tj], s, rh, rl);
#pragma unroll
        for (int ti = 0; ti < 2; ++ti) {
          const int off = (32 * ti + lc) * kBP * 2;
          const bf16x8 th = frag_row(Tbh + off, 32 * tj + 16 * s, h2);
          const bf16x8 tl = frag_row(Tbl + off, 32 * tj + 16 * s, h2);
          Dl[ti] = mma(tl, rh, mma(th, rl, mma(th, rh, Dl[ti])));
        }
      }
    // ---- 7. O = diag(2^G) Q M0 + (P o Q K^T) Delta
    if constexpr (OUT) {
#pragma unroll
    for (int ti = 0; ti < 2; ++ti)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const float4 g4 = ldf4((const lchar*)(eG + 32 * ti + 8 * r4 + 4 * h2));
        O[ti][4 * r4 + 0] *= g4.x;
        O[ti][4 * r4 + 1] *= g4.y;
        O[ti][4 * r4 + 2] *= g4.z;
        O[ti][4 * r4 + 3] *= g4.w;
      }
#pragma unroll
    for (int tj = 0; tj < 2; ++tj)
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        bf16x8 dh, dlo;
        split8(Dl[tj], s, dh, dlo);
#pragma unroll
        for (int ti = 0; ti < 2; ++ti) {
          const int off = (32 * ti + lc) * kBP * 2;
          const bf16x8 ph = frag_row(Ph + off, 32 * tj + 16 * s, h2);
          const bf16x8 pl = frag_row(Pl + off, 32 * tj + 16 * s, h2);
          O[ti] = mma(pl, dh, mma(ph, dlo, mma(ph, dh, O[ti])));
        }
      }
    lds_barrier();   // every wave is done with T diag(beta): O goes where A and T were
#pragma unroll
    for (int ti = 0; ti < 2; ++ti)
#pragma unroll
      for (int r = 0; r < 16; ++r) Os[(32 * ti + acc_row(r, lane)) * OP + col] = O[ti][r];
    }
    // ---- 8. M = 2^{G_C} M0 + K^T diag(2^{G_C - G}) Delta (K^T by transposed reads)
    const float eGC = eG[kC - 1];
#pragma unroll
    for (int tj = 0; tj < 2; ++tj)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const float4 e4 = ldf4((const lchar*)(eD + 32 * tj + 8 * r4 + 4 * h2));
        Dl[tj][4 * r4 + 0] *= e4.x;
        Dl[tj][4 * r4 + 1] *= e4.y;
        Dl[tj][4 * r4 + 2] *= e4.z;
        Dl[tj][4 * r4 + 3] *= e4.w;
      }
#pragma unroll
    for (int td = 0; td < NT; ++td)
#pragma unroll
      for (int r = 0; r < 16; ++r) M[td][r] *= eGC;
#pragma unroll
    for (int tj = 0; tj < 2; ++tj)
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        bf16x8 dh, dlo;
        split8(Dl[tj], s, dh, dlo);
#pragma unroll
        for (int td = 0; td < NT; ++td) {
          const int k0 = 32 * tj + 16 * s;
          const uint2 x0 = tr4(Ks, KP, k0, 32 * td), x1 = tr4(Ks, KP, k0 + 8, 32 * td);
          const bf16x8 ka = as_bf16x8(make_uint4(x0.x, x0.y, x1.x, x1.y));
          M[td] = mma(ka, dlo, mma(ka, dh, M[td]));
        }
      }
    lds_barrier();   // the output rows are complete; every wave is done with T
    // ---- 9. y = o / sqrt(mean(o^2) + eps) * w * SiLU(z): NW lanes per row,
    // 32 columns each
    if constexpr (OUT) {
      const int row = tid / NW, part = tid % NW;
      const float* orow = Os + row * OP + 32 * part;
      float ov[32];
      float ss = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float4 v = ldf4((const lchar*)(orow + 4 * e));
        ov[4 * e] = v.x; ov[4 * e + 1] = v.y; ov[4 * e + 2] = v.z; ov[4 * e + 3] = v.w;
        ss = fmaf(v.x, v.x, fmaf(v.y, v.y, fmaf(v.z, v.z, fmaf(v.w, v.w, ss))));
      }
#pragma unroll
      for (int off = 1; off < NW; off <<= 1) ss += __shfl_xor(ss, off);
      const float inv = __builtin_amdgcn_rsqf(ss / (float)DV + a.eps);
      if (row < n) {
        uint16_t* yrow = static_cast<uint16_t*>(a.Y) + (c0 + row) * ((int64_t)a.H_v * DV) + (int64_t)head * DV + 32 * part;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint4 z8 = ld16(Zs + (row * VP + 32 * part + 8 * e) * 2);
          const uint32_t zw[4] = {z8.x, z8.y, z8.z, z8.w};
          uint32_t yw[4];
#pragma unroll
          for (int p = 0; p < 4; ++p) {
            const int c = 8 * e + 2 * p;
            const float w0 = nws[32 * part + c], w1 = nws[32 * part + c + 1];
            yw[p] = pack_bf16x2(ov[c] * inv * w0 * silu(lo_f(zw[p])), ov[c + 1] * inv * w1 * silu(hi_f(zw[p])));
          }
          *reinterpret_cast<uint4*>(yrow + 8 * e) = make_uint4(yw[0], yw[1], yw[2], yw[3]);
        }
      }
    }
    lds_barrier();   // the next chunk's staging overwrites K, Q, V, Z; A overwrites the output rows
  }

  float* out = st_out + state_base;
#pragma unroll
  for (int td = 0; td < NT; ++td)
#pragma unroll
    for (int r = 0; r < 16; ++r) out[(size_t)(32 * td + acc_row(r, lane)) * DV + col] = M[td][r];
}

template <int D>
hipError_t run_output(const OutputArgs& a, hipStream_t s) {
  const int64_t units = (int64_t)a.n_seg * a.H_v;
  if (units == 0) return hipSuccess;
  hipLaunchKernelGGL((gdn_chunk_kernel<D, D, true, OutputArgs>), dim3((unsigned)units), dim3(OutCfg<D, D, true>::THREADS),
                     0, s, a);
  return hipGetLastError();
}

template <int DK, int DV>
hipError_t run_state(const ScanArgs& a, hipStream_t s) {
  const int64_t units = (int64_t)a.n_seg * a.n_layers * a.H_v;
  if (units == 0) return hipSuccess;
  hipLaunchKernelGGL((gdn_chunk_kernel<DK, DV, false, ScanArgs>), dim3((unsigned)units),
                     dim3(OutCfg<DK, DV, false>::THREADS), 0, s, a);
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

hipError_t launch_chunk_state(int d_k, int d_v, const ScanArgs& a, hipStream_t s) {
  if (d_k == 96 && d_v == 192) return run_state<96, 192>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace sr
