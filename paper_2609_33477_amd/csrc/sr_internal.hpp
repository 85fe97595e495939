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

// ------------------------------- fused projection + conv + gates (bf16 path)
// Per packed row: position inside its segment, rows left in the segment
// (this one included) and the segment's slot id (< 0: sentinel).
struct RowInfo {
  int32_t pos, rem, slot, seg;
};

struct ProjConvArgs {
  const void* A;        // anchors [T][K] bf16
  int64_t T;
  int32_t K;
  int32_t N;            // projection width C_kv + 2 H_v (columns k | v | a | b)
  int32_t n_wseg;
  WeightSeg seg[4];
  const RowInfo* info;  // [T]
  const void* conv_w;   // [C_kv][w]
  int32_t conv_bf16;    // conv_w dtype: 1 bf16, 0 fp32
  int32_t w;
  const float* a_log;
  const float* dt_bias;
  int32_t C_k, C_kv, H_v;
  float eps;
  void* Kbuf;           // [H_k][T][d] bf16
  void* Vbuf;           // [H_v][T][d] bf16
  float* Gbuf;          // [H_v][T] log2 alpha per row
  float* Bbuf;          // [H_v][T] beta
  void* tail;           // [slots][c_tail][w-1] or nullptr
  int32_t tail_bf16;
  int32_t c_tail;
  int32_t tail_kv_off;
  const int32_t* err;   // the call's table-check flag: non-zero = write nothing
};

hipError_t launch_row_info(const int32_t* cu, const int32_t* slot_ids, int32_t n_seg, RowInfo* info,
                           const int32_t* err, hipStream_t s);
hipError_t launch_proj_conv(int weight_dtype, int d_head, const ProjConvArgs& a, hipStream_t s);

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
  float* Gbuf;        // [H_v][T] ln alpha per row
  float* Bbuf;        // [H_v][T] beta
  void* tail;         // [slots][c_tail][w-1] or nullptr
  int32_t c_tail;
  int32_t tail_kv_off;  // first k channel inside the tail (q channels precede)
  const int32_t* err;   // the call's table-check flag: non-zero = write nothing
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
  const int32_t* err;   // the call's table-check flag: non-zero = write nothing
};

hipError_t launch_tail(int anchor_dtype, int weight_dtype, int tail_dtype, const TailArgs& a,
                       hipStream_t s);

// ------------------------------------------------------------ chunked scan
constexpr int kScanMaxLayers = 32;

struct ScanArgs {
  const void* Kbuf;     // layer l at Kbuf + l * kv_layer_stride elements: [H_k][T][d]
  const void* Vbuf;     // [H_v][T][d]
  const float* Gbuf;    // layer l at + l * g_layer_stride: [H_v][T]; per-row log decay:
                        // ln alpha (fp32 path) or log2 alpha (bf16 path)
  const float* Bbuf;
  int64_t k_layer_stride, v_layer_stride, g_layer_stride;
  int64_t T;
  const int32_t* cu;
  const int32_t* slot_ids;
  int32_t n_seg;
  int32_t H_k, H_v;
  int32_t n_layers;     // layers in this launch (<= kScanMaxLayers)
  const int32_t* err;   // the call's table-check flag: non-zero = write nothing
  const float* state_in[kScanMaxLayers];
  float* state_out[kScanMaxLayers];
};

hipError_t launch_scan(int op_dtype, int d_head, const ScanArgs& a, hipStream_t s);
hipError_t launch_scan_bf16(int d_head, const ScanArgs& a, hipStream_t s);
// per-head-decay recurrence: M = 2^{G_L} M_0 + K^T diag(beta 2^{G_L - G}) V (bf16 path)
hipError_t launch_decay_state(int d_head, const ScanArgs& a, hipStream_t s);

// ------------------------------------------------------ varlen table check
// One workgroup: writes 0 or a mask of sr_varlen_error bits to *flag and
// *status (either may be null).
hipError_t launch_validate(const int32_t* cu, const int32_t* slot_ids, int32_t n_seg, int64_t T, int32_t n_slots,
                           int32_t* flag, int32_t* status, hipStream_t s);

// ----------------------------------------------------------- launch timing
// Runs launch(ctx) on stream s under the library's per-kind timing and
// failed-launch bookkeeping (sr_kernel_timing_*, sr_last_hip_error).
hipError_t timed_launch(int kind, hipStream_t s, hipError_t (*launch)(void*), void* ctx);

// Records a failed HIP call of kernel kind `kind` for sr_last_hip_error
// (no-op for hipSuccess); returns e.
hipError_t note_error(int kind, hipError_t e);

template <typename F>
hipError_t timed_call(int kind, hipStream_t s, F&& f) {
  return timed_launch(kind, s, [](void* c) { return (*static_cast<F*>(c))(); }, &f);
}

}  // namespace sr
