// Fused short causal depthwise conv + SiLU + key L2 norm + decay/erase gates,
// and the conv tail (Appendix A: the conv state is the last w-1 inputs of the
// q, k, v channels).
//
// conv_gate_kernel: one wave per (row block, head); each lane owns d/64 (or one)
// channels of the head and walks the block's rows, keeping the previous w-1
// raw projection values in registers, so every projection element is read
// from HBM once (plus a (w-1)-row halo per block).  History is masked at
// segment starts: replay has no inputs before its first row.  Key heads are
// L2-normalised with a wave reduction.  The last y-block of the grid computes
// the per-(row, value head) gates:
//   g = log alpha = -exp(A_log) * softplus(a + dt_bias),  beta = sigmoid(b).
// Outputs are head-major ([H][T][d], [H][T]) so the scan reads each 64-row
// chunk of a head as one contiguous block.
//
// tail_kernel (fp32 anchors): per (segment, 64 channels), the q projections
// of the segment's last w-1 rows as dot products (W_q is used nowhere else),
// and zeros at positions before the segment's first row (every channel); the
// k | v channels of existing rows are written with k and v.  With bf16
// anchors the tail is computed inside the fused projection's grid.
#include "sr_device.hpp"
#include "tail_q.hpp"

#include <type_traits>

namespace sr {
namespace {

constexpr int kRowsPerBlock = 64;
constexpr int kConvThreads = 256;

__device__ __forceinline__ int segment_of_row(const int32_t* cu, int n_seg, int64_t t) {
  // Largest b with cu[b] <= t (skips empty segments): cu[b] <= t < cu[b+1].
  int lo = 0, hi = n_seg;  // answer in [0, n_seg)
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (cu[mid] <= t) lo = mid; else hi = mid;
  }
  return lo;
}

__device__ __forceinline__ float silu(float y) { return y / (1.f + expf(-y)); }
__device__ __forceinline__ float softplus(float x) { return fmaxf(x, 0.f) + log1pf(expf(-fabsf(x))); }
__device__ __forceinline__ float sigmoid(float x) { return 1.f / (1.f + expf(-x)); }

// One block per (64-row block, head), and one more per row block for the
// gates.  Rows run in parallel: a wave takes RPW rows of its head at a time
// (lane = CPL channels of one row), each lane reading the w raw rows its conv
// needs, so no row waits for the one before it; a key's sum of squares is
// reduced over the LPH lanes of its row.
template <typename OUT, typename CW, typename TT, int DH>
__global__ __launch_bounds__(kConvThreads) void conv_gate_kernel(ConvGateArgs a) {
  if (a.err && *a.err) return;   // the call's table check failed: write nothing
  constexpr int CPL = DH >= 64 ? DH / 64 : 1;   // channels per lane
  constexpr int LPH = DH / CPL;                   // lanes per head row
  constexpr int RPW = 64 / LPH;                   // rows per wave and pass
  constexpr int WAVES = kConvThreads / 64;
  constexpr int PASSES = kRowsPerBlock / (WAVES * RPW);
  constexpr int WMAX = 4;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int64_t r0 = (int64_t)blockIdx.x * kRowsPerBlock;
  const int64_t r1 = min(a.T, r0 + kRowsPerBlock);
  const int n_heads = a.H_k + a.H_v;
  const int C_kv = n_heads * DH;

  if ((int)blockIdx.y == n_heads) {
    // ---- gates: thread -> (head, row), rows fastest: ln alpha and beta per row
    const int rows = (int)(r1 - r0);
    for (int idx = tid; idx < rows * a.H_v; idx += kConvThreads) {
      const int h = idx / rows;
      const int64_t t = r0 + idx % rows;
      const float av = a.P[t * a.ldp + C_kv + h];
      const float bv = a.P[t * a.ldp + C_kv + a.H_v + h];
      a.Gbuf[(int64_t)h * a.T + t] = -expf(a.a_log[h]) * softplus(av + a.dt_bias[h]);
      a.Bbuf[(int64_t)h * a.T + t] = sigmoid(bv);
    }
    return;
  }

  const int head = blockIdx.y;
  const bool is_k = head < a.H_k;
  const int sub = lane % LPH;
  const int c0 = head * DH + sub * CPL;   // channel of the lane's first value
  const int w = a.w;
  float taps[CPL][WMAX];
#pragma unroll
  for (int q = 0; q < CPL; ++q)
#pragma unroll
    for (int i = 0; i < WMAX; ++i) taps[q][i] = (i < w) ? Elem<CW>::load(a.conv_w, (int64_t)(c0 + q) * w + i) : 0.f;
  void* dst = is_k ? a.Kbuf : a.Vbuf;
  const int hh = is_k ? head : head - a.H_k;

#pragma unroll
  for (int ps = 0; ps < PASSES; ++ps) {
    const int64_t t = r0 + (ps * WAVES + wid) * RPW + lane / LPH;
    const bool live = t < r1;
    int64_t s0 = 0, s1 = 0;
    int slot = -1;
    if (live) {
      const int b = segment_of_row(a.cu, a.n_seg, t);
      s0 = a.cu[b];
      s1 = a.cu[b + 1];
      slot = a.slot_ids ? a.slot_ids[b] : b;
    }
    // raw[d][q]: row t - d (zero before the segment's first row)
    float raw[WMAX][CPL];
#pragma unroll
    for (int d = 0; d < WMAX; ++d)
#pragma unroll
      for (int q = 0; q < CPL; ++q)
        raw[d][q] = (live && d < w && t - d >= s0) ? a.P[(t - d) * a.ldp + c0 + q] : 0.f;
    float act[CPL], ss = 0.f;
#pragma unroll
    for (int q = 0; q < CPL; ++q) {
      float y = 0.f;
#pragma unroll
      for (int d = 0; d < WMAX; ++d)
        if (d < w) y = fmaf(taps[q][w - 1 - d], raw[d][q], y);
      act[q] = silu(y);
      ss = fmaf(act[q], act[q], ss);
    }
    if (is_k) {
#pragma unroll
      for (int off = LPH / 2; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
      const float inv = 1.f / sqrtf(ss + a.eps);
#pragma unroll
      for (int q = 0; q < CPL; ++q) act[q] *= inv;
    }
    if (live) {
      const int64_t base = ((int64_t)hh * a.T + t) * DH + sub * CPL;
#pragma unroll
      for (int q = 0; q < CPL; ++q) Elem<OUT>::store(dst, base + q, act[q]);
      if (a.tail && slot >= 0 && t >= s1 - (w - 1)) {
        const int pos = (int)(t - (s1 - (w - 1)));
#pragma unroll
        for (int q = 0; q < CPL; ++q)
          Elem<TT>::store(a.tail, ((int64_t)slot * a.c_tail + a.tail_kv_off + c0 + q) * (w - 1) + pos, raw[0][q]);
      }
    }
  }
}

template <typename OUT, typename CW, typename TT, int DH>
hipError_t run_conv(const ConvGateArgs& a, hipStream_t s) {
  if (a.T == 0) return hipSuccess;
  static_assert(kRowsPerBlock % ((kConvThreads / 64) * (64 / (DH / (DH >= 64 ? DH / 64 : 1)))) == 0, "row passes");
  const int n_heads = a.H_k + a.H_v;
  dim3 grid((unsigned)((a.T + kRowsPerBlock - 1) / kRowsPerBlock), (unsigned)(n_heads + 1));
  hipLaunchKernelGGL((conv_gate_kernel<OUT, CW, TT, DH>), grid, dim3(kConvThreads), 0, s, a);
  return hipGetLastError();
}

// Heads whose key and value widths differ (Appendix A: OLMo-Hybrid's
// d_k = 96, d_v = 192): one wave per (row block, head), lane l owning
// channels l, l + 64, ... of its head, walking the block's rows as above; a
// key head's sum of squares is reduced over the wave.  G is written as
// log2 alpha, the convention of the chunk kernel that reads it.
template <typename OUT, typename CW, typename TT, int DK, int DV>
__global__ __launch_bounds__(kConvThreads) void conv_gate_rect_kernel(ConvGateArgs a) {
  if (a.err && *a.err) return;   // the call's table check failed: write nothing
  constexpr int QMAX = ((DK > DV ? DK : DV) + 63) / 64;   // channels per lane, at most
  constexpr int WMAX = 4;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int64_t r0 = (int64_t)blockIdx.x * kRowsPerBlock;
  const int64_t r1 = min(a.T, r0 + kRowsPerBlock);
  const int n_heads = a.H_k + a.H_v;
  const int C_kv = a.H_k * DK + a.H_v * DV;

  if ((int)blockIdx.y == (int)gridDim.y - 1) {
    // ---- gates: thread -> (head, row), rows fastest: log2 alpha and beta per row
    const int rows = (int)(r1 - r0);
    for (int idx = tid; idx < rows * a.H_v; idx += kConvThreads) {
      const int h = idx / rows;
      const int64_t t = r0 + idx % rows;
      const float av = a.P[t * a.ldp + C_kv + h];
      const float bv = a.P[t * a.ldp + C_kv + a.H_v + h];
      a.Gbuf[(int64_t)h * a.T + t] = -expf(a.a_log[h]) * softplus(av + a.dt_bias[h]) * 1.4426950408889634f;
      a.Bbuf[(int64_t)h * a.T + t] = sigmoid(bv);
    }
    return;
  }

  const int head = blockIdx.y * (kConvThreads / 64) + wid;
  if (head >= n_heads) return;                     // wave-uniform; the kernel has no block barrier
  const bool is_k = head < a.H_k;
  const int DH = is_k ? DK : DV;
  const int hh = is_k ? head : head - a.H_k;
  const int c0 = is_k ? head * DK : a.H_k * DK + hh * DV;   // first channel of the head
  const int w = a.w;

  float taps[QMAX][WMAX];
#pragma unroll
  for (int q = 0; q < QMAX; ++q) {
    const int ch = lane + 64 * q;
#pragma unroll
    for (int i = 0; i < WMAX; ++i)
      taps[q][i] = (ch < DH && i < w) ? Elem<CW>::load(a.conv_w, (int64_t)(c0 + ch) * w + i) : 0.f;
  }
  // prev[j][q] = raw value at row t-1-j
  float prev[WMAX - 1][QMAX];
#pragma unroll
  for (int j = 0; j < WMAX - 1; ++j)
#pragma unroll
    for (int q = 0; q < QMAX; ++q) {
      const int ch = lane + 64 * q;
      const int64_t t = r0 - 1 - j;
      prev[j][q] = (ch < DH && j < w - 1 && t >= 0) ? a.P[t * a.ldp + c0 + ch] : 0.f;
    }

  int b = segment_of_row(a.cu, a.n_seg, r0);
  int64_t s0 = a.cu[b], s1 = a.cu[b + 1];
  int slot = a.slot_ids ? a.slot_ids[b] : b;
  void* dst = is_k ? a.Kbuf : a.Vbuf;

  for (int64_t t = r0; t < r1; ++t) {
    while (t >= s1) {
      ++b;
      s0 = a.cu[b];
      s1 = a.cu[b + 1];
      slot = a.slot_ids ? a.slot_ids[b] : b;
    }
    float raw[QMAX], act[QMAX];
    float ss = 0.f;
#pragma unroll
    for (int q = 0; q < QMAX; ++q) {
      const int ch = lane + 64 * q;
      raw[q] = ch < DH ? a.P[t * a.ldp + c0 + ch] : 0.f;
      float y = taps[q][w - 1] * raw[q];
#pragma unroll
      for (int j = 0; j < WMAX - 1; ++j)
        if (j < w - 1 && t - 1 - j >= s0) y = fmaf(taps[q][w - 2 - j], prev[j][q], y);
      act[q] = silu(y);
      ss = fmaf(act[q], act[q], ss);
    }
    if (is_k) {
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
      const float inv = 1.f / sqrtf(ss + a.eps);
#pragma unroll
      for (int q = 0; q < QMAX; ++q) act[q] *= inv;
    }
    const int64_t base = ((int64_t)hh * a.T + t) * DH;
    const bool tail_row = a.tail && slot >= 0 && t >= s1 - (w - 1);
    const int pos = (int)(t - (s1 - (w - 1)));
#pragma unroll
    for (int q = 0; q < QMAX; ++q) {
      const int ch = lane + 64 * q;
      if (ch < DH) {
        Elem<OUT>::store(dst, base + ch, act[q]);
        if (tail_row) Elem<TT>::store(a.tail, ((int64_t)slot * a.c_tail + a.tail_kv_off + c0 + ch) * (w - 1) + pos, raw[q]);
      }
    }
#pragma unroll
    for (int j = WMAX - 2; j > 0; --j)
#pragma unroll
      for (int q = 0; q < QMAX; ++q) prev[j][q] = prev[j - 1][q];
#pragma unroll
    for (int q = 0; q < QMAX; ++q) prev[0][q] = raw[q];
  }
}

template <typename OUT, typename CW, typename TT, int DK, int DV>
hipError_t run_conv_rect(const ConvGateArgs& a, hipStream_t s) {
  if (a.T == 0) return hipSuccess;
  const int n_heads = a.H_k + a.H_v;
  constexpr int HPB = kConvThreads / 64;   // heads per block
  dim3 grid((unsigned)((a.T + kRowsPerBlock - 1) / kRowsPerBlock), (n_heads + HPB - 1) / HPB + 1);
  hipLaunchKernelGGL((conv_gate_rect_kernel<OUT, CW, TT, DK, DV>), grid, dim3(kConvThreads), 0, s, a);
  return hipGetLastError();
}

template <typename OUT, typename CW, typename TT>
hipError_t conv_by_head(int d, const ConvGateArgs& a, hipStream_t s) {
  if (a.d_k != a.d_v) {
    if constexpr (std::is_same<OUT, bf16_t>::value) {
      if (a.d_k == 96 && a.d_v == 192) return run_conv_rect<OUT, CW, TT, 96, 192>(a, s);
    }
    return hipErrorInvalidValue;
  }
  switch (d) {
    case 32: return run_conv<OUT, CW, TT, 32>(a, s);
    case 64: return run_conv<OUT, CW, TT, 64>(a, s);
    case 128: return run_conv<OUT, CW, TT, 128>(a, s);
  }
  return hipErrorInvalidValue;
}

template <typename OUT, typename CW>
hipError_t conv_by_tail(int tail_dtype, int d, const ConvGateArgs& a, hipStream_t s) {
  if (tail_dtype == SR_F32) return conv_by_head<OUT, CW, float>(d, a, s);
  if (tail_dtype == SR_BF16) return conv_by_head<OUT, CW, bf16_t>(d, a, s);
  return hipErrorInvalidValue;
}

// ------------------------------------------------------------------ tail
constexpr int kTailThreads = 256;
constexpr int kTailChannels = 4;   // one channel per wave: the channels' loads run in parallel

// 8 consecutive elements starting at element i, as fp32.
template <typename T>
__device__ __forceinline__ void load8(const void* p, int64_t i, float* out);
template <>
__device__ __forceinline__ void load8<float>(const void* p, int64_t i, float* out) {
  const float4* q = reinterpret_cast<const float4*>(static_cast<const float*>(p) + i);
  const float4 x = q[0], y = q[1];
  out[0] = x.x; out[1] = x.y; out[2] = x.z; out[3] = x.w;
  out[4] = y.x; out[5] = y.y; out[6] = y.z; out[7] = y.w;
}

template <typename TA, typename TW, typename TT>
__global__ __launch_bounds__(kTailThreads) void tail_kernel(TailArgs a) {
  if (a.err && *a.err) return;   // the call's table check failed: write nothing
  constexpr int WMAX = 4;
  const int b = blockIdx.x;
  const int slot = a.slot_ids ? a.slot_ids[b] : b;
  if (slot < 0) return;
  const int64_t s0 = a.cu[b], s1 = a.cu[b + 1];
  const int w1 = a.w - 1;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int cb = blockIdx.y * kTailChannels;
  const int ce = min(a.c_tail, cb + kTailChannels);

  // zero-fill positions that precede the segment's first row
  for (int idx = tid; idx < (ce - cb) * w1; idx += kTailThreads) {
    const int c = cb + idx / w1, pos = idx % w1;
    if (s1 - w1 + pos < s0) Elem<TT>::store(a.tail, ((int64_t)slot * a.c_tail + c) * w1 + pos, 0.f);
  }
  if (cb >= a.c_q) return;

  // q channels: dot products of W_q rows with the last w-1 anchor rows
  const int per_wave = kTailChannels / (kTailThreads / 64);
  for (int ci = 0; ci < per_wave; ++ci) {
    const int c = cb + wid * per_wave + ci;
    if (c >= min(ce, a.c_q)) break;
    float acc[WMAX - 1] = {0.f, 0.f, 0.f};
    for (int k = lane * 8; k < a.D; k += 64 * 8) {
      float wv[8];
      load8<TW>(a.w_q, (int64_t)c * a.D + k, wv);
#pragma unroll
      for (int pos = 0; pos < WMAX - 1; ++pos) {
        const int64_t t = s1 - w1 + pos;
        if (pos < w1 && t >= s0) {
          float xv[8];
          load8<TA>(a.anchors, t * a.D + k, xv);
#pragma unroll
          for (int j = 0; j < 8; ++j) acc[pos] = fmaf(xv[j], wv[j], acc[pos]);
        }
      }
    }
#pragma unroll
    for (int pos = 0; pos < WMAX - 1; ++pos)
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) acc[pos] += __shfl_xor(acc[pos], off);
    if (lane == 0) {
      const float scale = std::is_same<TW, fp8_t>::value ? Elem<bf16_t>::load(a.s_q, c) : 1.f;
      for (int pos = 0; pos < w1; ++pos)
        if (s1 - w1 + pos >= s0)
          Elem<TT>::store(a.tail, ((int64_t)slot * a.c_tail + c) * w1 + pos, acc[pos] * scale);
    }
  }
}

template <typename TA, typename TW, typename TT>
hipError_t run_tail(const TailArgs& a, hipStream_t s) {
  if (a.n_seg == 0 || a.w < 2 || a.c_tail == 0) return hipSuccess;
  dim3 grid(a.n_seg, (a.c_tail + kTailChannels - 1) / kTailChannels);
  hipLaunchKernelGGL((tail_kernel<TA, TW, TT>), grid, dim3(kTailThreads), 0, s, a);
  return hipGetLastError();
}

template <typename TT>
hipError_t tail_by_input(int ad, int wd, const TailArgs& a, hipStream_t s) {
  if (ad == SR_F32 && wd == SR_F32) return run_tail<float, float, TT>(a, s);
  return hipErrorInvalidValue;
}

// The q-tail blocks of tail_q.hpp in a grid of their own (bf16 anchors on a
// path without the fused projection)
template <typename TW>
__global__ __launch_bounds__(64 * kTqWaves) void tail_q_kernel(TailArgs a) {
  if (a.err && *a.err) return;   // the call's table check failed: write nothing
  __shared__ __attribute__((aligned(1024))) char smem[kTqLds];
  tail_q_block<TW>(a, blockIdx.x, blockIdx.y, smem);
}

}  // namespace

hipError_t launch_conv_gate(int op_dtype, int conv_dtype, int tail_dtype, int d_head,
                            const ConvGateArgs& a, hipStream_t s) {
  if (op_dtype == SR_F32) {
    if (conv_dtype == SR_F32) return conv_by_tail<float, float>(tail_dtype, d_head, a, s);
    if (conv_dtype == SR_BF16) return conv_by_tail<float, bf16_t>(tail_dtype, d_head, a, s);
  } else if (op_dtype == SR_BF16) {
    if (conv_dtype == SR_F32) return conv_by_tail<bf16_t, float>(tail_dtype, d_head, a, s);
    if (conv_dtype == SR_BF16) return conv_by_tail<bf16_t, bf16_t>(tail_dtype, d_head, a, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_tail(int anchor_dtype, int weight_dtype, int tail_dtype, const TailArgs& a,
                       hipStream_t s) {
  if (anchor_dtype == SR_BF16) {
    if (a.n_seg == 0 || a.w < 2 || a.c_tail == 0) return hipSuccess;
    const dim3 grid(tail_q_grid_x(a), tail_q_grid_y(a));
    if (weight_dtype == SR_BF16) hipLaunchKernelGGL((tail_q_kernel<bf16_t>), grid, dim3(64 * kTqWaves), 0, s, a);
    else if (weight_dtype == SR_FP8_E4M3) hipLaunchKernelGGL((tail_q_kernel<fp8_t>), grid, dim3(64 * kTqWaves), 0, s, a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
  }
  if (tail_dtype == SR_F32) return tail_by_input<float>(anchor_dtype, weight_dtype, a, s);
  if (tail_dtype == SR_BF16) return tail_by_input<bf16_t>(anchor_dtype, weight_dtype, a, s);
  return hipErrorInvalidValue;
}

}  // namespace sr
