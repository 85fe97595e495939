// Row RMSNorm of a replayed block (group replay chaining, Section 4.1: a
// pre-norm block normalises its input rows before the mixer and again before
// the MLP).  One wave per row of D elements: 8-element vectors, the sum of
// squares reduced over the wave, then x / sqrt(mean(x^2) + eps) * w rounded to
// bf16 (the operand of the next GEMM).  With a copy target the fp32 input row
// is also written there (the group-entry anchors start the fp32 residual
// stream).  HBM-bound: 2 or 4 bytes in, 2 (+4) out per element.
#include "sr_device.hpp"

namespace sr {
namespace {

constexpr int kRows = 4;   // waves (rows) per block

__device__ __forceinline__ void load8(const void* x, bool bf16, int64_t i, float* v) {
  if (bf16) {
    const uint4 u = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(x) + i);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[2 * e] = __uint_as_float(w[e] << 16);
      v[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
    }
  } else {
    const float4 a = *reinterpret_cast<const float4*>(static_cast<const float*>(x) + i);
    const float4 b = *reinterpret_cast<const float4*>(static_cast<const float*>(x) + i + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
}

template <int VPL>   // 8-element vectors per lane
__global__ __launch_bounds__(64 * kRows) void rmsnorm_kernel(RmsNormArgs a) {
  if (a.err && *a.err) return;   // the call's table check failed: write nothing
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * kRows + (threadIdx.x >> 6);
  if (t >= a.T) return;
  const int D = a.D;
  const int64_t base = t * D;
  float x[VPL][8];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    const int c = (j * 64 + lane) * 8;
    if (c < D) {
      load8(a.x, a.in_bf16 != 0, base + c, x[j]);
#pragma unroll
      for (int e = 0; e < 8; ++e) ss = fmaf(x[j][e], x[j][e], ss);
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off);
  const float inv = __builtin_amdgcn_rsqf(ss / (float)D + a.eps);
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    const int c = (j * 64 + lane) * 8;
    if (c < D) {
      float w[8];
      load8(a.w, true, c, w);
      uint4 o;
      o.x = pack_bf16x2(x[j][0] * inv * w[0], x[j][1] * inv * w[1]);
      o.y = pack_bf16x2(x[j][2] * inv * w[2], x[j][3] * inv * w[3]);
      o.z = pack_bf16x2(x[j][4] * inv * w[4], x[j][5] * inv * w[5]);
      o.w = pack_bf16x2(x[j][6] * inv * w[6], x[j][7] * inv * w[7]);
      *reinterpret_cast<uint4*>(static_cast<uint16_t*>(a.out) + base + c) = o;
      if (a.copy) {
        *reinterpret_cast<float4*>(a.copy + base + c) = make_float4(x[j][0], x[j][1], x[j][2], x[j][3]);
        *reinterpret_cast<float4*>(a.copy + base + c + 4) = make_float4(x[j][4], x[j][5], x[j][6], x[j][7]);
      }
    }
  }
}

}  // namespace

hipError_t launch_rmsnorm(const RmsNormArgs& a, hipStream_t s) {
  if (a.T == 0) return hipSuccess;
  if (a.D % 8 || a.D > 64 * 8 * 16) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((a.T + kRows - 1) / kRows));
  const int vpl = (a.D + 511) / 512;
  if (vpl <= 4) hipLaunchKernelGGL(rmsnorm_kernel<4>, grid, dim3(64 * kRows), 0, s, a);
  else if (vpl <= 8) hipLaunchKernelGGL(rmsnorm_kernel<8>, grid, dim3(64 * kRows), 0, s, a);
  else hipLaunchKernelGGL(rmsnorm_kernel<16>, grid, dim3(64 * kRows), 0, s, a);
  return hipGetLastError();
}

}  // namespace sr
