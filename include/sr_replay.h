/*
 * sr_replay.h -- C ABI of the SuffixReplay state-reconstruction library
 * (hand-written HIP for gfx950 / MI355X).
 *
 * SuffixReplay rebuilds a linear-attention layer's recurrent state at a cached
 * page boundary by replaying a bounded suffix of that layer's retained input
 * hidden states ("anchors") from a zero state (paper Section 1, Eq. 1-2;
 * Section 4.3 for the per-hit anchor contract).  Replay writes the rebuilt
 * recurrent state and the short-convolution state into the request's
 * preallocated slots (Section 5.2), and batches many hits into one varlen
 * execution with device-side segment boundaries and a sentinel slot id for
 * padding segments (Section 5.2, "Batched replay").
 *
 * For one Gated DeltaNet layer and one segment of L anchor rows h_1..h_L the
 * library computes (Section 2.1, Eq. recurrence, with the layer's projections):
 *   k|v|a|b = W_{k|v|a|b} h_t                       (projection, fp32 accumulate)
 *   k, v    = SiLU(causal depthwise conv_w(k|v))    (zero history before h_1)
 *   k       = k / sqrt(|k|^2 + l2_eps)              (per key head)
 *   alpha_t = exp(-exp(A_log) softplus(a_t + dt_bias)),  beta_t = sigmoid(b_t)
 *   S_t     = alpha_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T, S_0 = 0
 * and emits M = S_L^T per value head, plus the conv tail (Appendix A): the raw
 * pre-conv projections of the last w-1 rows, channels q | k | v.
 * Value head h reads key head floor(h * H_k / H_v).
 *
 * Conventions
 *  - Every tensor pointer is a DEVICE pointer owned by the caller; the library
 *    allocates nothing.  Scratch comes from the caller's workspace, sized by
 *    sr_replay_workspace_size().
 *  - Matrices are row-major.  Weights are [out][in = d_model] (nn.Linear).
 *  - sr_replay_state() only enqueues work on `stream` (a hipStream_t; NULL is
 *    the default stream) and never synchronises with the host, so it can be
 *    captured into a HIP graph.  Completion is stream-ordered.
 *  - Argument and shape errors are detected on the host before any launch and
 *    return a status with nothing written.  SR_ERR_HIP means a launch failed;
 *    outputs are then undefined.  A caller treats any non-SR_OK status as a
 *    cache miss (the fail-closed rule of Section 5.2).  The library never
 *    aborts or prints.
 *  - The device tables are checked on the device, first thing in the call
 *    (cu_seqlens[0] = 0, non-decreasing, cu_seqlens[n_segments] = t_total;
 *    live slot ids < n_slots and distinct).  If the check fails, every later
 *    kernel of the call exits without writing anything, and the reason (a
 *    mask of sr_varlen_error bits) goes to the optional device word
 *    varlen_status and to the first 4 bytes of the workspace; the caller
 *    treats a non-zero mask as a cache miss.
 *  - Outputs must not alias inputs or the workspace.  Calls that share a
 *    workspace must be ordered on one stream.
 */
#ifndef SR_REPLAY_H
#define SR_REPLAY_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum sr_status {
  SR_OK = 0,
  SR_ERR_NULL_ARG = 1,          /* a required pointer is NULL                  */
  SR_ERR_BAD_SHAPE = 2,         /* a size is out of the supported range        */
  SR_ERR_UNSUPPORTED_DTYPE = 3, /* dtype or dtype combination not supported    */
  SR_ERR_WORKSPACE_TOO_SMALL = 4,
  SR_ERR_MISALIGNED = 5,        /* a tensor pointer is not 16-byte aligned     */
  SR_ERR_HIP = 6                /* a HIP launch or runtime call failed         */
} sr_status;

typedef enum sr_dtype {
  SR_F32 = 0,
  SR_BF16 = 1,
  SR_FP8_E4M3 = 2               /* OCP FP8 E4M3 (bias 7, max 448)              */
} sr_dtype;

/* Shape and storage types of one linear-attention layer.
 *  d_model     anchor width D; multiple of 64, 64 <= D <= 16384
 *  n_k_heads   H_k >= 1;  n_v_heads H_v, a multiple of H_k, H_v <= 128
 *  d_k, d_v    head dims: d_k = d_v in {32, 64, 128}, or d_k = 96 with
 *              d_v = 192 (OLMo-Hybrid-7B, Appendix A; BF16 anchors and the
 *              Gated DeltaNet recurrence only, SR_ERR_UNSUPPORTED_DTYPE
 *              otherwise); any other pair is SR_ERR_BAD_SHAPE
 *  conv_width  w in 1..4 (the paper's models use 4)
 *  l2_eps      key-norm epsilon (> 0)
 *  dtypes      supported (anchor, weight) pairs: (F32, F32), (BF16, BF16),
 *              (BF16, FP8_E4M3).  conv_dtype is F32 or BF16, tail_dtype F32 or
 *              BF16.  F32 anchors run the whole path in fp32 arithmetic; BF16
 *              anchors run bf16 MFMA with fp32 accumulation and an fp32 state. */
typedef struct sr_shape {
  int32_t d_model;
  int32_t n_k_heads;
  int32_t n_v_heads;
  int32_t d_k;
  int32_t d_v;
  int32_t conv_width;
  float l2_eps;
  int32_t anchor_dtype;
  int32_t weight_dtype;
  int32_t conv_dtype;
  int32_t tail_dtype;
  int32_t recurrence;   /* sr_recurrence; 0 (the zero-initialised default) = Gated DeltaNet */
} sr_shape;

/* The state update (Section 2.1, Eq. recurrence; both share the layer's
 * projections, conv, key norm and gates):
 *  SR_RECURRENCE_GDN    S_t = alpha_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T
 *  SR_RECURRENCE_DECAY  S_t = alpha_t S_{t-1} + beta_t v_t k_t^T: the per-head decay
 *                       without erase that the paper names for Mamba2; BF16
 *                       anchors only (SR_ERR_UNSUPPORTED_DTYPE otherwise) */
typedef enum sr_recurrence {
  SR_RECURRENCE_GDN = 0,
  SR_RECURRENCE_DECAY = 1
} sr_recurrence;

/* Tensors of one layer (all device pointers).  T = t_total, D = d_model.
 *  anchors    [T][D] anchor_dtype: the packed replay suffixes of all segments
 *  w_k        [H_k*d_k][D]   w_v [H_v*d_v][D]   w_a, w_b [H_v][D]   weight_dtype
 *  w_q        [H_k*d_k][D] or NULL.  Only feeds the q part of the conv tail.
 *  s_k, s_v, s_a, s_b, s_q
 *             FP8 weights only: bf16 per-output-channel scales ([rows]); the
 *             effective weight is diag(s) Q.  Ignored (may be NULL) otherwise.
 *  conv_w     [H_k*d_k + H_v*d_v][w] conv_dtype: k channels then v channels;
 *             tap w-1 multiplies the current row.
 *  a_log, dt_bias   [H_v] fp32
 *  state_in   NULL (the method: replay starts from zero) or
 *             [n_slots][H_v][d_k][d_v] fp32 initial state read at each live
 *             segment's slot.
 *  state_out  [n_slots][H_v][d_k][d_v] fp32; element [s][h][i][j] is
 *             S_L[j][i] of value head h (M = S^T).  Written for live slots only.
 *  tail_out   NULL (no conv tail) or [n_slots][C_tail][w-1] tail_dtype with
 *             C_tail = (w_q ? 2*H_k*d_k : H_k*d_k) + H_v*d_v, channels q | k | v,
 *             positions oldest -> newest; positions before a segment's first
 *             row are zero.  Written for live slots only. */
typedef struct sr_layer {
  const void* anchors;
  const void* w_k;
  const void* w_v;
  const void* w_a;
  const void* w_b;
  const void* w_q;
  const void* s_k;
  const void* s_v;
  const void* s_a;
  const void* s_b;
  const void* s_q;
  const void* conv_w;
  const float* a_log;
  const float* dt_bias;
  const float* state_in;
  float* state_out;
  void* tail_out;
} sr_layer;

/* Bytes of one slot's recurrent state: H_v * d_k * d_v * 4 (Appendix A,
 * B_rec).  0 if `shape` is NULL. */
size_t sr_state_bytes(const sr_shape* shape);

/* Bytes of one slot's conv tail: C_tail * (w-1) * sizeof(tail_dtype), with q
 * channels counted when with_q != 0 (Appendix A, B_conv for a bf16 tail).
 * 0 if `shape` is NULL. */
size_t sr_conv_tail_bytes(const sr_shape* shape, int32_t with_q);

/* Workspace bytes sr_replay_state() needs for `n_layers` layers of `t_total`
 * packed anchor rows each.  Host-only; writes *bytes. */
sr_status sr_replay_workspace_size(const sr_shape* shape, int32_t n_layers,
                                   int64_t t_total, size_t* bytes);

/* Replay `n_segments` packed suffixes through `n_layers` independent layers
 * (Section 5.2, batched replay) and write each live segment's final state and
 * conv tail into its slot of every layer.
 *  layers       host array of n_layers sr_layer (1 <= n_layers <= 256); all
 *               layers share `shape` and the segment boundaries
 *  n_segments   >= 0 (0 is a no-op)
 *  t_total      total packed rows per layer, 0 <= t_total < 2^31
 *  cu_seqlens   device int32 [n_segments+1], segment b = rows
 *               [cu_seqlens[b], cu_seqlens[b+1])
 *  slot_ids     device int32 [n_segments] or NULL (slot b for segment b);
 *               a negative id is the sentinel: that segment's state, tail and
 *               initial state are neither read nor written
 *  n_slots      slots of every layer's state_out / tail_out / state_in
 *               (0 <= n_slots <= SR_MAX_SLOTS); live slot ids must be below it
 *  varlen_status  NULL or a device int32 that receives the table check's
 *               result (0, or a mask of sr_varlen_error bits) when the call
 *               runs
 *  workspace    device scratch of >= sr_replay_workspace_size() bytes,
 *               256-byte aligned
 *  stream       hipStream_t (NULL = default stream)
 * A segment with zero rows yields the initial state (zero, or state_in) and a
 * zero tail. */
sr_status sr_replay_state(const sr_shape* shape, int32_t n_layers, const sr_layer* layers,
                          int32_t n_segments, int64_t t_total, const int32_t* cu_seqlens,
                          const int32_t* slot_ids, int32_t n_slots, int32_t* varlen_status,
                          void* workspace, size_t workspace_bytes, void* stream);

/* Reasons the device check of the varlen tables fails (Section 5.2: a bad
 * input is a cache miss, never a corrupt write). */
typedef enum sr_varlen_error {
  SR_VARLEN_BAD_START = 1,       /* cu_seqlens[0] != 0                          */
  SR_VARLEN_NOT_MONOTONE = 2,    /* cu_seqlens[b + 1] < cu_seqlens[b]           */
  SR_VARLEN_BAD_TOTAL = 4,       /* cu_seqlens[n_segments] != t_total           */
  SR_VARLEN_SLOT_RANGE = 8,      /* a live slot id >= n_slots                   */
  SR_VARLEN_SLOT_DUPLICATE = 16  /* two live segments share a slot id           */
} sr_varlen_error;

/* Largest n_slots the device check accepts (its slot bitmap lives in LDS). */
#define SR_MAX_SLOTS (1 << 19)

/* The device check that sr_replay_state runs first, on its own: reads
 * cu_seqlens [n_segments + 1] and slot_ids [n_segments] (or NULL: identity)
 * and writes 0 or a mask of sr_varlen_error bits to the device int32
 * *status, stream-ordered.  For debugging a serving system's tables.
 * SR_ERR_BAD_SHAPE if n_segments < 1, t_total < 0 or n_slots is outside
 * 0..SR_MAX_SLOTS; SR_ERR_NULL_ARG if cu_seqlens or status is NULL. */
sr_status sr_validate_varlen(const int32_t* cu_seqlens, const int32_t* slot_ids, int32_t n_segments,
                             int64_t t_total, int32_t n_slots, int32_t* status, void* stream);

/* The same check on host arrays (host pointers, no device work): writes the
 * mask to *mask.  Argument errors as sr_validate_varlen. */
sr_status sr_validate_varlen_host(const int32_t* cu_seqlens, const int32_t* slot_ids, int32_t n_segments,
                                  int64_t t_total, int32_t n_slots, int32_t* mask);

/* Largest workspace sr_replay_state_noalloc() can serve (128 MiB: e.g. 4096
 * packed rows of one Qwen3.5-4B or Qwen3.6-27B linear layer). */
#define SR_NOALLOC_SCRATCH_BYTES (128u << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the replay
 * of sr_replay_state() with the same arguments minus the workspace, which
 * comes from a library-owned device array of SR_NOALLOC_SCRATCH_BYTES per GPU
 * (held until the process ends).  Calls no hipMalloc, hipFree or allocating
 * library routine.
 *  - SR_ERR_WORKSPACE_TOO_SMALL, with nothing written, when
 *    sr_replay_workspace_size() for these arguments exceeds
 *    SR_NOALLOC_SCRATCH_BYTES.
 *  - Every call on a GPU shares that GPU's array: calls that overlap on one
 *    GPU race, so calls on one device must be ordered (one stream, or
 *    events).  The array keeps the last call's contents; a call never reads
 *    scratch it has not written.
 *  - The first call on a device resolves the array's device address
 *    (SR_ERR_HIP if that fails); later calls reuse it. */
sr_status sr_replay_state_noalloc(const sr_shape* shape, int32_t n_layers, const sr_layer* layers,
                                  int32_t n_segments, int64_t t_total, const int32_t* cu_seqlens,
                                  const int32_t* slot_ids, int32_t n_slots, int32_t* varlen_status,
                                  void* stream);

/* Kernels the library launches, as indexed by sr_kernel_timing_read(). */
typedef enum sr_kernel_kind {
  SR_KERNEL_PROJ_GEMM = 0,   /* anchor projection (MFMA), fp32 path           */
  SR_KERNEL_CONV_GATE = 1,   /* conv + SiLU + key norm + gates + k|v tail,
                                fp32 path                                     */
  SR_KERNEL_TAIL = 2,        /* q part of the conv tail + zero fill           */
  SR_KERNEL_GDN_SCAN = 3,    /* chunked state accumulation                    */
  SR_KERNEL_PROJ_CONV = 4,   /* projection fused with conv, SiLU, key norm,
                                gates and the k|v tail (bf16 / fp8 path); one
                                launch covers up to 4 layers of a call        */
  SR_KERNEL_ROW_INFO = 5,    /* per-row segment position and slot; runs in
                                the table check's launch (SR_KERNEL_VALIDATE)
                                and is never launched on its own            */
  SR_KERNEL_ANCHOR_COMPACT = 6,  /* sidecar: prefill compaction (sr_sidecar.h)  */
  SR_KERNEL_ANCHOR_WRITE = 7,    /* sidecar: indexed copy into the blocks       */
  SR_KERNEL_ANCHOR_SEQLENS = 8,  /* sidecar: segment offsets of a gather        */
  SR_KERNEL_ANCHOR_GATHER = 9,   /* sidecar: gather of the replay anchors       */
  SR_KERNEL_DECAY_STATE = 10,    /* per-head-decay state (SR_RECURRENCE_DECAY)  */
  SR_KERNEL_GRAPH = 11,          /* graph replay: capture, launch, parameter
                                    kernel, anchor fetch (sr_replay_graph.h)    */
  SR_KERNEL_VALIDATE = 12,       /* device check of the varlen tables           */
  SR_KERNEL_RMSNORM = 13,        /* group replay: block RMSNorm (sr_group.h)    */
  SR_KERNEL_GDN_OUTPUT = 14,     /* group replay: states and gated outputs      */
  SR_KERNEL_GEMM_RESID = 15,     /* group replay: output / down projection      */
  SR_KERNEL_GEMM_SWIGLU = 16,    /* group replay: MLP gate and up projections   */
  SR_KERNEL_KINDS = 17
} sr_kernel_kind;

/* Benchmark instrumentation (not needed by the replay itself).  While
 * enabled, sr_replay_state() and the sidecar calls of sr_sidecar.h record a
 * HIP event pair around every kernel launch on the caller's stream (creating
 * events on first use).
 * sr_kernel_timing_read() waits for the recorded events, adds each pair's
 * elapsed time to ms[kind] and its count to launches[kind] (arrays of
 * SR_KERNEL_KINDS, zeroed by the call), then discards the records.
 * Not thread-safe; not for use under graph capture. */
sr_status sr_kernel_timing_enable(int32_t enable);
sr_status sr_kernel_timing_read(double* ms, int64_t* launches);
/* The kinds recorded while timing is enabled: bit k of `mask` for kind k
 * (default: every kind).  Launches of other kinds run without events, so a
 * benchmark can time one kernel live without bracketing the others. */
sr_status sr_kernel_timing_kinds(uint32_t mask);

/* Diagnostics for SR_ERR_HIP: the HIP error code (hipError_t) and the
 * sr_kernel_kind of the calling thread's most recent failed launch inside a
 * library call, and hipGetErrorString() of that code (static storage).
 * *hip_error is 0 and *kernel_kind -1 if no launch has failed on this thread.
 * Any output pointer may be NULL.  Always returns SR_OK. */
sr_status sr_last_hip_error(int32_t* hip_error, int32_t* kernel_kind, const char** message);

/* Static, NUL-terminated description of a status code. */
const char* sr_status_str(sr_status status);

#ifdef __cplusplus
}
#endif

#endif /* SR_REPLAY_H */
