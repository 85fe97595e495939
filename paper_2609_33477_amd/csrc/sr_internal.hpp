// Host/device interface between the C ABI (sr_api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sr_replay.h"

namespace sr {

// ----------------------------------------------------------------- projection
// C[m][n] = sum_k A[m][k] * W(n)[k] * scale(n) for n < N, where output column
// n comes from row (n - n0) of the weight segment that covers it.
struct WeightSeg {
  const void* ptr;    // [n1 - n0][K]
  const void* scale;  // bf16 [n1 - n0] (fp8 weights only)
  int32_t n0, n1;
};

struct GemmArgs {
  const void* A;      // [M][K]
  int64_t M;
  int32_t K;
  int32_t N;
  int32_t n_seg;
  WeightSeg seg[4];
  float* C;           // [M][ldc]
  int64_t ldc;
};

hipError_t launch_proj_gemm(int anchor_dtype, int weight_dtype, const GemmArgs& a, hipStream_t s);

// --------------------------------------------------- conv, activations, gates
struct ConvGateArgs {
  const float* P;     // [T][ldp] projection, columns k | v | a | b
  int64_t ldp;
  int64_t T;
  const int32_t* cu;
  const int32_t* slot_ids;
  int32_t n_seg;
  const void* conv_w; // [C_kv][w]
  int32_t w;
  const float* a_log;
  const float* dt_bias;
  int32_t H_k, H_v;
  float eps;
  void* Kbuf;         // [H_k][T][d] operand dtype
  void* Vbuf;         // [H_v][T][d]
  float* Gbuf;        // [H_v][T]: g_mode 0 -> ln alpha per row; 1 -> log2 alpha summed
                      // from the start of the row's 16-row sub-chunk (sub-chunks
                      // start at the segment start and every 16 rows after it)
  int32_t g_mode;
  float* Bbuf;        // [H_v][T] beta
  void* tail;         // [slots][c_tail][w-1] or nullptr
  int32_t c_tail;
  int32_t tail_kv_off;  // first k channel inside the tail (q channels precede)
};

hipError_t launch_conv_gate(int op_dtype, int conv_dtype, int tail_dtype, int d_head,
                            const ConvGateArgs& a, hipStream_t s);

// ------------------------------------------------- conv tail: q part + zeros
struct TailArgs {
  const void* anchors;  // [T][D]
  int32_t D;
  const void* w_q;      // [c_q][D] or nullptr
  const void* s_q;      // bf16 [c_q] (fp8 only)
  int32_t c_q;          // q channels in the tail (0 without w_q)
  const int32_t* cu;
  const int32_t* slot_ids;
  int32_t n_seg;
  int32_t w;
  void* tail;           // [slots][c_tail][w-1]
  int32_t c_tail;
};

hipError_t launch_tail(int anchor_dtype, int weight_dtype, int tail_dtype, const TailArgs& a,
                       hipStream_t s);

// ------------------------------------------------------------ chunked scan
constexpr int kScanMaxLayers = 32;

struct ScanArgs {
  const void* Kbuf;     // layer l at Kbuf + l * kv_layer_stride elements: [H_k][T][d]
  const void* Vbuf;     // [H_v][T][d]
  const float* Gbuf;    // layer l at + l * g_layer_stride: [H_v][T]
  const float* Bbuf;
  int64_t k_layer_stride, v_layer_stride, g_layer_stride;
  int64_t T;
  const int32_t* cu;
  const int32_t* slot_ids;
  int32_t n_seg;
  int32_t H_k, H_v;
  int32_t n_layers;     // layers in this launch (<= kScanMaxLayers)
  const float* state_in[kScanMaxLayers];
  float* state_out[kScanMaxLayers];
};

hipError_t launch_scan(int op_dtype, int d_head, const ScanArgs& a, hipStream_t s);
hipError_t launch_scan_bf16(int d_head, const ScanArgs& a, hipStream_t s);

}  // namespace sr
