// Anchor projection GEMM: P[T][N] = anchors[T][D] * [W_k; W_v; W_a; W_b]^T.
//
// The projection of the replayed anchors is the only dense contraction on the
// replay path (the update's key, value and gate inputs are linear maps of the
// layer input, Section 2.1), so it runs on MFMA: bf16 x bf16 with
// v_mfma_f32_32x32x16_bf16, fp8 (E4M3) weights converted exactly to bf16
// while they are staged into LDS with the per-output-channel scale applied to
// the fp32 accumulator (W8A16), and an fp32 variant on v_mfma_f32_32x32x2f32.
//
// Block tile BM x BN, K step BK, double-buffered LDS (one barrier per step)
// fed from registers that prefetch the next K step during the MFMA work.
#include "sr_device.hpp"

#include <type_traits>

namespace sr {
namespace {

template <typename TA, typename TB, int BM_, int BN_, int BK_, int WM_, int WN_>
struct GemmCfg {
  using OP = typename std::conditional<std::is_same<TA, float>::value, float, bf16_t>::type;
  using MF = Mfma<OP>;
  static constexpr int BM = BM_, BN = BN_, BK = BK_, WM = WM_, WN = WN_;
  static constexpr int THREADS = WM * WN * 64;
  static constexpr int TM = BM / WM, TN = BN / WN;
  static constexpr int FM = TM / 32, FN = TN / 32;
  static constexpr int EB = std::is_same<OP, float>::value ? 4 : 2;   // LDS element bytes
  static constexpr int LDK = BK + 16 / EB;                             // padded row pitch (elements)
  static constexpr int VA = 16 / Elem<TA>::bytes;                      // A elements per 16-byte load
  static constexpr int VB = 16 / Elem<TB>::bytes;
  static constexpr int A_LOADS = BM * BK / VA / THREADS;
  static constexpr int B_LOADS = BN * BK / VB / THREADS;
  static constexpr int STAGE_BYTES = (BM + BN) * LDK * EB;
  static_assert(BM * BK % (VA * THREADS) == 0, "A tile split");
  static_assert(BN * BK % (VB * THREADS) == 0, "B tile split");
  static_assert(TM % 32 == 0 && TN % 32 == 0, "wave tile");
};

// Store one 16-byte global chunk (VB elements of TB) into LDS as operand type.
template <typename TB>
__device__ __forceinline__ void stage_b(char* dst, const uint4& v);

template <>
__device__ __forceinline__ void stage_b<bf16_t>(char* dst, const uint4& v) {
  *reinterpret_cast<uint4*>(dst) = v;
}
template <>
__device__ __forceinline__ void stage_b<float>(char* dst, const uint4& v) {
  *reinterpret_cast<uint4*>(dst) = v;
}
template <>
__device__ __forceinline__ void stage_b<fp8_t>(char* dst, const uint4& v) {
  // 16 fp8 -> 16 bf16 (32 bytes), exact.
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  uint32_t o[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t x = w[i];
    o[2 * i] = e4m3_to_bf16_bits(x & 0xffu) | (e4m3_to_bf16_bits((x >> 8) & 0xffu) << 16);
    o[2 * i + 1] = e4m3_to_bf16_bits((x >> 16) & 0xffu) | (e4m3_to_bf16_bits(x >> 24) << 16);
  }
  reinterpret_cast<uint4*>(dst)[0] = make_uint4(o[0], o[1], o[2], o[3]);
  reinterpret_cast<uint4*>(dst)[1] = make_uint4(o[4], o[5], o[6], o[7]);
}

template <typename OP>
__device__ __forceinline__ typename Mfma<OP>::frag lds_frag(const char* base, int row, int k, int ldk);

template <>
__device__ __forceinline__ bf16x8 lds_frag<bf16_t>(const char* base, int row, int k, int ldk) {
  return as_bf16x8(*reinterpret_cast<const uint4*>(base + ((size_t)row * ldk + k) * 2));
}
template <>
__device__ __forceinline__ float lds_frag<float>(const char* base, int row, int k, int ldk) {
  return *reinterpret_cast<const float*>(base + ((size_t)row * ldk + k) * 4);
}

template <typename CFG, typename TA, typename TB>
__global__ __launch_bounds__(CFG::THREADS) void proj_gemm_kernel(GemmArgs g) {
  using OP = typename CFG::OP;
  using MF = typename CFG::MF;
  constexpr int BM = CFG::BM, BN = CFG::BN, BK = CFG::BK;
  constexpr int LDK = CFG::LDK, EB = CFG::EB;
  __shared__ __attribute__((aligned(16))) char smem[2 * CFG::STAGE_BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = tid >> 6;
  const int wm = wid / CFG::WN;
  const int wn = wid % CFG::WN;
  const int64_t m0 = (int64_t)blockIdx.y * BM;
  const int n0 = blockIdx.x * BN;

  // Per-thread global source rows (fixed over the K loop).
  const char* a_src[CFG::A_LOADS];
  int a_dst[CFG::A_LOADS];
  constexpr int A_CPR = BK / CFG::VA;  // chunks per row
#pragma unroll
  for (int i = 0; i < CFG::A_LOADS; ++i) {
    const int c = tid + i * CFG::THREADS;
    const int r = c / A_CPR, kc = c % A_CPR;
    const int64_t m = m0 + r;
    a_src[i] = (m < g.M) ? static_cast<const char*>(g.A) + (m * g.K + kc * CFG::VA) * Elem<TA>::bytes
                         : nullptr;
    a_dst[i] = (r * LDK + kc * CFG::VA) * EB;
  }
  const char* b_src[CFG::B_LOADS];
  int b_dst[CFG::B_LOADS];
  constexpr int B_CPR = BK / CFG::VB;
#pragma unroll
  for (int i = 0; i < CFG::B_LOADS; ++i) {
    const int c = tid + i * CFG::THREADS;
    const int r = c / B_CPR, kc = c % B_CPR;
    const int n = n0 + r;
    const char* p = nullptr;
    if (n < g.N) {
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        if (s < g.n_seg && n >= g.seg[s].n0 && n < g.seg[s].n1)
          p = static_cast<const char*>(g.seg[s].ptr) +
              ((int64_t)(n - g.seg[s].n0) * g.K + kc * CFG::VB) * Elem<TB>::bytes;
      }
    }
    b_src[i] = p;
    b_dst[i] = CFG::BM * LDK * EB + (r * LDK + kc * CFG::VB) * EB;
  }

  uint4 ra[CFG::A_LOADS], rb[CFG::B_LOADS];
  auto load_regs = [&](int kt) {
    const int64_t koff_a = (int64_t)kt * BK * Elem<TA>::bytes;
    const int64_t koff_b = (int64_t)kt * BK * Elem<TB>::bytes;
#pragma unroll
    for (int i = 0; i < CFG::A_LOADS; ++i)
      ra[i] = a_src[i] ? *reinterpret_cast<const uint4*>(a_src[i] + koff_a) : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < CFG::B_LOADS; ++i)
      rb[i] = b_src[i] ? *reinterpret_cast<const uint4*>(b_src[i] + koff_b) : make_uint4(0, 0, 0, 0);
  };
  auto store_regs = [&](int buf) {
    char* base = smem + buf * CFG::STAGE_BYTES;
#pragma unroll
    for (int i = 0; i < CFG::A_LOADS; ++i) *reinterpret_cast<uint4*>(base + a_dst[i]) = ra[i];
#pragma unroll
    for (int i = 0; i < CFG::B_LOADS; ++i) stage_b<TB>(base + b_dst[i], rb[i]);
  };

  f32x16 acc[CFG::FM][CFG::FN];
#pragma unroll
  for (int i = 0; i < CFG::FM; ++i)
#pragma unroll
    for (int j = 0; j < CFG::FN; ++j) acc[i][j] = zero16();

  const int KT = g.K / BK;
  load_regs(0);
  store_regs(0);
  __syncthreads();

  const int fr = lane & 31;
  const int fk = (lane >> 5) * MF::HALF;
  for (int kt = 0; kt < KT; ++kt) {
    if (kt + 1 < KT) load_regs(kt + 1);
    const char* As = smem + (kt & 1) * CFG::STAGE_BYTES;
    const char* Bs = As + BM * LDK * EB;
#pragma unroll
    for (int ks = 0; ks < BK / MF::K; ++ks) {
      typename MF::frag fa[CFG::FM], fb[CFG::FN];
#pragma unroll
      for (int i = 0; i < CFG::FM; ++i)
        fa[i] = lds_frag<OP>(As, wm * CFG::TM + i * 32 + fr, ks * MF::K + fk, LDK);
#pragma unroll
      for (int j = 0; j < CFG::FN; ++j)
        fb[j] = lds_frag<OP>(Bs, wn * CFG::TN + j * 32 + fr, ks * MF::K + fk, LDK);
#pragma unroll
      for (int i = 0; i < CFG::FM; ++i)
#pragma unroll
        for (int j = 0; j < CFG::FN; ++j) MF::mma(acc[i][j], fa[i], fb[j]);
    }
    if (kt + 1 < KT) store_regs((kt + 1) & 1);
    __syncthreads();
  }

  // Epilogue: per-column scale (fp8 weights), bounds-checked fp32 store.
#pragma unroll
  for (int j = 0; j < CFG::FN; ++j) {
    const int n = n0 + wn * CFG::TN + j * 32 + fr;
    if (n >= g.N) continue;
    float scale = 1.f;
    if (std::is_same<TB, fp8_t>::value) {
#pragma unroll
      for (int s = 0; s < 4; ++s)
        if (s < g.n_seg && n >= g.seg[s].n0 && n < g.seg[s].n1)
          scale = Elem<bf16_t>::load(g.seg[s].scale, n - g.seg[s].n0);
    }
#pragma unroll
    for (int i = 0; i < CFG::FM; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t m = m0 + wm * CFG::TM + i * 32 + acc_row(r, lane);
        if (m < g.M) g.C[m * g.ldc + n] = acc[i][j][r] * scale;
      }
    }
  }
}

template <typename CFG, typename TA, typename TB>
hipError_t run(const GemmArgs& g, hipStream_t s) {
  if (g.M == 0) return hipSuccess;
  dim3 grid((g.N + CFG::BN - 1) / CFG::BN, (unsigned)((g.M + CFG::BM - 1) / CFG::BM));
  hipLaunchKernelGGL((proj_gemm_kernel<CFG, TA, TB>), grid, dim3(CFG::THREADS), 0, s, g);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_proj_gemm(int anchor_dtype, int weight_dtype, const GemmArgs& g, hipStream_t s) {
  if (anchor_dtype == SR_F32 && weight_dtype == SR_F32)
    return run<GemmCfg<float, float, 64, 64, 32, 2, 2>, float, float>(g, s);
  if (anchor_dtype == SR_BF16 && weight_dtype == SR_BF16)
    return run<GemmCfg<bf16_t, bf16_t, 256, 256, 64, 2, 4>, bf16_t, bf16_t>(g, s);
  if (anchor_dtype == SR_BF16 && weight_dtype == SR_FP8_E4M3)
    return run<GemmCfg<bf16_t, fp8_t, 256, 256, 64, 2, 4>, bf16_t, fp8_t>(g, s);
  return hipErrorInvalidValue;
}

}  // namespace sr
