// Per-head-decay state accumulation (the Mamba2 form named in Section 2.1: a
// scalar decay per head and no erase), bf16 operands on gfx950.
//
// With S_t = alpha_t S_{t-1} + beta_t v_t k_t^T, the unrolled form (Section
// 2.1, Eq. unrolled) gives the final state directly:
//   M = S_L^T = 2^{G_L} M_0 + K^T diag(c) V,   c_t = beta_t 2^{G_L - G_t},
// with G the segment prefix of log2 alpha.  No row waits for another, so the
// state is one weighted reduction over the segment's rows: no triangular
// solve and no sequential chunk carry.
//
// One workgroup (4 waves) per (segment, layer, value head), longest segments
// first.  Rows go 64 at a time from the segment's end backwards, so the
// exponent of a row's weight is a running sum of the log decays after it
// (small terms added in order, never the difference of two large sums).  Per
// chunk: every wave turns log2 alpha and beta into the weights c (a suffix
// scan over its 64 lanes); every thread scales its V vectors by c, rounds
// them to bf16 and writes K and cV to one of two LDS buffers (row pitch
// d + 16 elements, so the 4 rows a transposed read touches sit in distinct
// banks) while the previous chunk's products run on the other; the loads of
// the chunk two ahead are issued; each wave
// accumulates its share of the d x d output on v_mfma_f32_16x16x32_bf16,
// reading both operands down their rows with ds_read_b64_tr_b16.
#include "sr_device.hpp"
#include "sr_internal.hpp"

namespace sr {
namespace {

constexpr int kRows = 64;        // rows per chunk
constexpr int kThreads = 256;    // 4 waves

typedef __attribute__((address_space(3))) char lchar;
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

template <int D>
struct DCfg {
  static constexpr int P = D + 16;                 // LDS row pitch (bf16 elements)
  static constexpr int MAT = kRows * P * 2;        // bytes of one [64][P] matrix
  static constexpr int VPT = kRows * D / 8 / kThreads;   // 16-byte vectors per thread and matrix
  static constexpr int TI = D / 16;                // 16 x 16 output tiles per dimension
  static constexpr int NI = TI >= 4 ? TI / 4 : 1;  // tiles per wave: NI rows x NJ columns
  static constexpr int NJ = TI >= 4 ? TI : 1;
};

template <int D>
__global__ __launch_bounds__(kThreads, 2) void decay_state_kernel(ScanArgs a) {
  if (a.err && *a.err) return;   // the call's table check failed: write nothing
  using C = DCfg<D>;
  constexpr int P = C::P, VPT = C::VPT, NI = C::NI, NJ = C::NJ, VPR = D / 8;
  __shared__ __attribute__((aligned(16))) char smem[4 * C::MAT];   // two buffers of K and cV
  __shared__ float g_total;        // G_L, for the initial state
  __shared__ int sel;
  lchar* Ks = (lchar*)smem;
  lchar* Vs = Ks + C::MAT;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, j = lane & 15;

  // Consecutive blocks r and r + 8 land on one XCD: give them value heads 2k
  // and 2k + 1, which share a key head when H_v = 2 H_k.
  const int units = a.n_seg * a.n_layers * a.H_v;
  int u = blockIdx.x;
  if ((u | 15) < units) u = (u & ~15) + 2 * (u & 7) + ((u >> 3) & 1);
  const int head = u % a.H_v;
  const int layer = (u / a.H_v) % a.n_layers;
  const int b = segment_of_rank(a, u / (a.H_v * a.n_layers), &sel);
  const int slot = a.slot_ids ? a.slot_ids[b] : b;
  if (slot < 0) return;
  const int64_t s0 = a.cu[b], s1 = a.cu[b + 1];
  const int nch = (int)((s1 - s0 + kRows - 1) / kRows);
  const int hk = (head * a.H_k) / a.H_v;
  const uint16_t* Kp = static_cast<const uint16_t*>(a.Kbuf) + layer * a.k_layer_stride + (int64_t)hk * a.T * D;
  const uint16_t* Vp = static_cast<const uint16_t*>(a.Vbuf) + layer * a.v_layer_stride + (int64_t)head * a.T * D;
  const float* Gp = a.Gbuf + layer * a.g_layer_stride + (int64_t)head * a.T;
  const float* Bp = a.Bbuf + layer * a.g_layer_stride + (int64_t)head * a.T;

  // this thread's vectors: vector q = tid + 256 m is row q / VPR, columns
  // 8 (q % VPR) .. + 7 of a chunk.  Two register sets alternate, so a chunk's
  // loads are issued two chunks before it is staged.
  struct Regs {
    u32x4 k[VPT], v[VPT];
    float g, b;   // log2 alpha and beta of row `lane` (every wave holds them)
  };
  Regs ra, rb;
  auto load_chunk = [&](Regs& R, int n) {
    const int64_t base = s1 - (int64_t)kRows * (n + 1);   // row 0 of chunk n (may precede s0)
#pragma unroll
    for (int m = 0; m < VPT; ++m) {
      const int q = tid + kThreads * m;
      int64_t t = base + q / VPR;
      t = t < s0 ? s0 : t;   // rows before the segment get weight 0
      R.k[m] = *reinterpret_cast<const u32x4*>(Kp + t * D + 8 * (q % VPR));
      R.v[m] = *reinterpret_cast<const u32x4*>(Vp + t * D + 8 * (q % VPR));
    }
    const int64_t t = base + lane;
    const bool ok = t >= s0;
    R.g = ok ? Gp[t] : 0.f;
    R.b = ok ? Bp[t] : 0.f;
  };

  f32x4 acc[NI][NJ];
#pragma unroll
  for (int x = 0; x < NI; ++x)
#pragma unroll
    for (int y = 0; y < NJ; ++y) acc[x][y] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int it0 = C::TI >= 4 ? wid * NI : wid >> 1;   // first output tile row / column of this wave
  const int jt0 = C::TI >= 4 ? 0 : wid & 1;

  // Every wave computes the weights of the chunk it stages: c of row `lane`
  // from the suffix sums over the chunk; the rows of this thread's vectors
  // take theirs from the owning lane.
  float s_after = 0.f;   // sum of log2 alpha over the rows after the chunk being staged
  auto stage = [&](Regs& R, int buf) {
    float x = R.g;       // incl(r) = sum of g over rows >= r
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float y = __shfl_down(x, off, 64);
      if (lane + off < 64) x += y;
    }
    const float c_lane = R.b * __builtin_amdgcn_exp2f(s_after + (x - R.g));
    s_after += __shfl(x, 0, 64);
    lchar* Kd = Ks + buf * 2 * C::MAT;
    lchar* Vd = Kd + C::MAT;
#pragma unroll
    for (int m = 0; m < VPT; ++m) {
      const int q = tid + kThreads * m;
      const int r = q / VPR, off = (r * P + 8 * (q % VPR)) * 2;
      const float c = __shfl(c_lane, r, 64);
      const u32x4 v = R.v[m];
      u32x4 sv;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        sv[e] = pack_bf16x2(bf16_bits_to_f32(v[e] & 0xffffu) * c, bf16_bits_to_f32(v[e] >> 16) * c);
      *reinterpret_cast<__attribute__((address_space(3))) u32x4*>(Kd + off) = R.k[m];
      *reinterpret_cast<__attribute__((address_space(3))) u32x4*>(Vd + off) = sv;
    }
  };
  // M[i][jj] += sum_t K[t][i] cV[t][jj] over the chunk in buffer buf
  auto products = [&](int buf) {
    const lchar* Kb = Ks + buf * 2 * C::MAT;
    const lchar* Vb = Kb + C::MAT;
#pragma unroll
    for (int kk = 0; kk < kRows / 32; ++kk) {
      const int rowb = 32 * kk + 8 * g + (j >> 2);
      bf16x8 fa[NI], fb[NJ];
#pragma unroll
      for (int x = 0; x < NI; ++x) {
        const lchar* p = Kb + (rowb * P + 16 * (it0 + x) + 4 * (j & 3)) * 2;
        const uint2 lo = lds_tr4(p), hi = lds_tr4(p + 4 * P * 2);
        fa[x] = as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
      }
#pragma unroll
      for (int y = 0; y < NJ; ++y) {
        const lchar* p = Vb + (rowb * P + 16 * (jt0 + y) + 4 * (j & 3)) * 2;
        const uint2 lo = lds_tr4(p), hi = lds_tr4(p + 4 * P * 2);
        fb[y] = as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
      }
#pragma unroll
      for (int x = 0; x < NI; ++x)
#pragma unroll
        for (int y = 0; y < NJ; ++y) acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[x], fb[y], acc[x][y], 0, 0, 0);
    }
  };
  // Chunk n is staged into buffer n % 2 while the products of chunk n - 1 run
  // on the other buffer; one barrier per chunk.
  if (nch > 0) load_chunk(ra, 0);
  if (nch > 1) load_chunk(rb, 1);
  if (nch > 0) {
    stage(ra, 0);
    if (nch > 2) load_chunk(ra, 2);
  }
  __syncthreads();
  for (int n = 0; n < nch; n += 2) {
    // chunk n in buffer 0 (its products), chunk n + 1 from rb into buffer 1
    if (n + 1 < nch) {
      stage(rb, 1);
      if (n + 3 < nch) load_chunk(rb, n + 3);
    }
    products(0);
    __syncthreads();
    if (n + 1 < nch) {
      // chunk n + 1 in buffer 1, chunk n + 2 from ra into buffer 0
      if (n + 2 < nch) {
        stage(ra, 0);
        if (n + 4 < nch) load_chunk(ra, n + 4);
      }
      products(1);
      __syncthreads();
    }
  }
  if (tid == 0) g_total = s_after;
  __syncthreads();

  // M = acc + 2^{G_L} M_0; lane holds rows 4 g .. 4 g + 3 of column j of each tile
  const char* kargs = (const char*)__builtin_amdgcn_kernarg_segment_ptr();
  const float* st_in = *reinterpret_cast<const float* const*>(kargs + offsetof(ScanArgs, state_in) + sizeof(void*) * layer);
  float* st_out = *reinterpret_cast<float* const*>(kargs + offsetof(ScanArgs, state_out) + sizeof(void*) * layer);
  const size_t state_base = ((size_t)slot * a.H_v + head) * D * D;
  const float carry = __builtin_amdgcn_exp2f(g_total);
#pragma unroll
  for (int x = 0; x < NI; ++x)
#pragma unroll
    for (int y = 0; y < NJ; ++y)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const size_t idx = state_base + (size_t)(16 * (it0 + x) + 4 * g + r) * D + 16 * (jt0 + y) + j;
        float m = acc[x][y][r];
        if (st_in) m += carry * st_in[idx];
        st_out[idx] = m;
      }
}

template <int D>
hipError_t run(const ScanArgs& a, hipStream_t s) {
  const int64_t units = (int64_t)a.n_seg * a.n_layers * a.H_v;
  if (units == 0) return hipSuccess;
  hipLaunchKernelGGL((decay_state_kernel<D>), dim3((unsigned)units), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_decay_state(int d_head, const ScanArgs& a, hipStream_t s) {
  switch (d_head) {
    case 32: return run<32>(a, s);
    case 64: return run<64>(a, s);
    case 128: return run<128>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace sr
