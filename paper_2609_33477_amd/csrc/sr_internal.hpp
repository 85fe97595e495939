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
  int32_t tail_bf16;    // tail dtype (q-tail blocks of the fused projection): 1 bf16, 0 fp32
  int32_t c_tail;
  const int32_t* err;   // the call's table-check flag: non-zero = write nothing
};

// q-tail grid (bf16 anchors): x = 32-channel blocks of the q channels + 1
// block for the leading zeros of the others; y = 32-row blocks of the
// n_seg (w-1) tail rows.
__host__ __device__ inline int tail_q_grid_x(const TailArgs& a) { return (a.c_q + 31) / 32 + 1; }
__host__ __device__ inline int tail_q_grid_y(const TailArgs& a) { return (a.n_seg * (a.w - 1) + 31) / 32; }

struct ProjConvArgs {
  const void* A;        // anchors [T][K] bf16
  int64_t T;
  int32_t K;
  int32_t N;            // projection width: columns [q |] k | v [| z] | a | b
  int32_t n_wseg;
  WeightSeg seg[6];
  const RowInfo* info;  // [T]
  const void* conv_w;   // [C_kv][w]: taps of the conv columns ([q |] k | v)
  int32_t conv_bf16;    // conv_w dtype: 1 bf16, 0 fp32
  int32_t w;
  const float* a_log;
  const float* dt_bias;
  // column ranges: q [0, C_q), k [C_q, C_k), v [C_k, C_kv), z [C_kv, C_z),
  // a [C_z, C_z + H_v), b [C_z + H_v, N); C_q = 0 and C_z = C_kv without q / z
  int32_t C_q, C_k, C_kv, C_z, H_v;
  float eps;
  float q_scale;        // multiplies the normalised q (d^-1/2)
  void* Qbuf;           // [H_k][T][d] bf16 (with q columns)
  void* Zbuf;           // [H_v][T][d] bf16 (with z columns)
  void* Kbuf;           // [H_k][T][d] bf16
  void* Vbuf;           // [H_v][T][d] bf16
  float* Gbuf;          // [H_v][T] log2 alpha per row
  float* Bbuf;          // [H_v][T] beta
  void* tail;           // [slots][c_tail][w-1] or nullptr
  int32_t tail_bf16;
  int32_t c_tail;
  int32_t tail_kv_off;
  const int32_t* err;   // the call's table-check flag: non-zero = write nothing
  // q part of the conv tail and its leading zeros (bf16 anchors), run by
  // blocks appended to the projection's grid; tq_blocks = 0: none
  TailArgs tq;
  int32_t tq_blocks;
  // Heads whose key width k_real is below the kernel's head width D (the
  // rectangular-head variant; no q or z columns): each key head takes D
  // output columns, its last D - k_real zero, and Kbuf keeps that padded
  // [H_k][T][D] layout; value heads are v_head = 2 k_real columns wide and
  // stored as two halves padded the same way ([2 H_v][T][D], pads zero).
  // Weight segments, fp8 scales, conv taps and the tail are in the caller's
  // unpadded channel order.  0, 0 for square heads.
  int32_t k_real, v_head;
};

// The projections of up to kProjBatch layers of one call in one launch: every
// layer of a call has the same T and N, so the grid holds the tiles of all of
// them (a small batch leaves CUs idle in a launch of its own), then their
// q-tail blocks.
constexpr int kProjBatch = 4;
struct ProjConvBatch {
  ProjConvArgs layer[kProjBatch];   // layers 0 .. n_layers-1; T, K and N equal
  int32_t n_layers;
  int32_t tq_off[kProjBatch + 1];   // layer i's q-tail blocks: [tq_off[i], tq_off[i+1]) after the tiles
};

hipError_t launch_proj_conv(int weight_dtype, int d_head, const ProjConvBatch& b, hipStream_t s);
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
  // key and value head widths; d_k != d_v takes the one-head-per-wave kernel
  // (bf16 operands), whose G is log2 alpha (the chunk kernel's convention)
  int32_t d_k, d_v;
};

hipError_t launch_conv_gate(int op_dtype, int conv_dtype, int tail_dtype, int d_head,
                            const ConvGateArgs& a, hipStream_t s);

// fp32 anchors: per-segment dot products; bf16 anchors: the q-tail blocks on
// their own (the fused projection's grid carries them when it runs)
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
  int32_t k_pitch;      // elements per K row (0: d_k); rectangular heads: 128 (padded keys)
  // bf16 scan only: each value head runs as v_split units of D state
  // columns (0 or 1: one unit per head).  H_v and the V planes then count
  // units; G and beta stay per value head (unit / v_split), and the state of
  // value head h is [st_rows][st_pitch] fp32 of which unit h v_split + e
  // holds rows < st_rows, columns [e st_cols, (e + 1) st_cols).  0: D each.
  int32_t v_split, st_rows, st_cols, st_pitch;
};

hipError_t launch_scan(int op_dtype, int d_head, const ScanArgs& a, hipStream_t s);
hipError_t launch_scan_bf16(int d_head, const ScanArgs& a, hipStream_t s);
// per-head-decay recurrence: M = 2^{G_L} M_0 + K^T diag(beta 2^{G_L - G}) V (bf16 path)
hipError_t launch_decay_state(int d_head, const ScanArgs& a, hipStream_t s);

// ------------------------------------------ group replay: block GEMMs, norms
constexpr int kGemmResid = 0, kGemmSwiglu = 1;

// C = A B^T, A [M][K] bf16 row-major, B [N][K] bf16 (B2: the up weights of
// the SwiGLU mode, B the gate weights).  kGemmResid: C fp32 [M][ldc] += acc;
// kGemmSwiglu: C bf16 [M][ldc] = SiLU(A B^T) * (A B2^T), N = 2 * hidden.
struct BlockGemmArgs {
  const void* A;
  int64_t M;
  int32_t K, N;
  const void* B;
  const void* B2;
  void* C;
  int64_t ldc;
  const int32_t* err;
};
hipError_t launch_block_gemm(int mode, const BlockGemmArgs& a, hipStream_t s);

// Row RMSNorm: out[t] = bf16(x[t] / sqrt(mean(x[t]^2) + eps) * w) for x
// bf16 (in_bf16) or fp32 rows of D; copy (optional, fp32) receives x[t].
struct RmsNormArgs {
  const void* x;
  int32_t in_bf16;
  int64_t T;
  int32_t D;
  const void* w;       // bf16 [D]
  float eps;
  void* out;           // bf16 [T][D]
  float* copy;         // fp32 [T][D] or nullptr
  const int32_t* err;
};
hipError_t launch_rmsnorm(const RmsNormArgs& a, hipStream_t s);

// Chunked Gated DeltaNet with per-token outputs (one launch per layer):
// states as the scan kernels, and y = RMSNorm_head(o) * norm_w * SiLU(z),
// o_t = S_t q_t, into Y [T][H_v * d] bf16.
struct OutputArgs {
  const void* Qbuf;     // [H_k][T][d] bf16, q already scaled by d^-1/2
  const void* Kbuf;     // [H_k][T][d]
  const void* Vbuf;     // [H_v][T][d]
  const void* Zbuf;     // [H_v][T][d]
  const float* Gbuf;    // [H_v][T] log2 alpha
  const float* Bbuf;    // [H_v][T] beta
  int64_t T;
  const int32_t* cu;
  const int32_t* slot_ids;
  int32_t n_seg;
  int32_t H_k, H_v;
  const void* norm_w;   // bf16 [d]
  float eps;
  void* Y;              // [T][H_v * d] bf16
  float* state_out;     // [slots][H_v][d][d]
  const int32_t* err;
};
hipError_t launch_gdn_output(int d_head, const OutputArgs& a, hipStream_t s);
// State-only chunked scan of heads with d_k != d_v (bf16 operands, log2 alpha
// gates), the same chunk algebra as the output kernel; (d_k, d_v) = (96, 192)
hipError_t launch_chunk_state(int d_k, int d_v, const ScanArgs& a, hipStream_t s);

// ------------------------------------------------------ varlen table check
// One workgroup: writes 0 or a mask of sr_varlen_error bits to *flag and
// *status (either may be null).
hipError_t launch_validate(const int32_t* cu, const int32_t* slot_ids, int32_t n_seg, int64_t T, int32_t n_slots,
                           int32_t* flag, int32_t* status, hipStream_t s);
// the check and the rows' segment info for the fused projection, one launch
hipError_t launch_validate_rows(const int32_t* cu, const int32_t* slot_ids, int32_t n_seg, int64_t T,
                                int32_t n_slots, int32_t* flag, int32_t* status, RowInfo* info, hipStream_t s);

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
