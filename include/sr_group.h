/*
 * sr_group.h -- group replay chaining (part of libsr_replay).
 *
 * Section 4.1 stores one anchor per group of consecutive linear-attention
 * layers -- the hidden state entering the group -- and rebuilds every layer of
 * the group from it: each replayed layer's block output is the next layer's
 * input, and replay never crosses the full-attention layer that closes the
 * group (Appendix A: A = G - 1 stored anchors instead of one per linear
 * layer).  sr_replay_group rebuilds the recurrent state and conv tail of every
 * layer of one group, for a packed varlen batch of hits (Section 5.2,
 * "Batched replay"), from the group-entry anchors alone.
 *
 * A block is pre-norm around a Gated DeltaNet mixer (Section 2.1; Appendix A
 * for the state and conv shapes).  The paper prints none of the block's
 * algebra; the library computes, per row (eps = norm_eps):
 *   x  = RMSNorm(h) * ln_in                       (over d_model)
 *   q|k|v|z|a|b = W x;  q, k, v through the causal conv (taps conv_w, zero
 *        history before the segment) and SiLU; q and k L2-normalised per key
 *        head (l2_eps), q scaled by d_k^-1/2;  alpha, beta as sr_replay.h
 *   S_t = alpha_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T,  o_t = S_t q_t
 *   y  = RMSNorm(o) * norm_o * SiLU(z)            (per value head, over d_v)
 *   h1 = h + W_o y;   u = RMSNorm(h1) * ln_post
 *   h' = h1 + W_down (SiLU(W_gate u) * (W_up u))  (the next layer's input)
 * Value head h reads query and key head floor(h H_k / H_v).  The last layer's
 * block output is not formed (a full-attention layer follows).  The hidden
 * state between layers is kept in fp32; every GEMM operand is bf16 with fp32
 * accumulation.
 *
 * Conventions are those of sr_replay.h: device pointers owned by the caller,
 * a caller workspace (sr_group_workspace_size), stream-ordered and
 * graph-capturable, host checks before any launch, the device check of the
 * varlen tables first in the call (nothing is written if it fails).
 */
#ifndef SR_GROUP_H
#define SR_GROUP_H

#include <stddef.h>
#include <stdint.h>

#include "sr_replay.h"

#ifdef __cplusplus
extern "C" {
#endif

/* One block's tensors (device pointers, bf16 unless stated; D = d_model,
 * C_tail = 2 H_k d_k + H_v d_v):
 *  w_q, w_k  [H_k d_k][D]     w_v, w_z [H_v d_v][D]     w_a, w_b [H_v][D]
 *  conv_w    [C_tail][w] conv taps of the q | k | v channels (conv_dtype);
 *            tap w-1 multiplies the current row
 *  a_log, dt_bias  [H_v] fp32
 *  norm_o    [d_v] weight of the per-head output norm
 *  w_o       [D][H_v d_v]
 *  ln_in, ln_post  [D] norm weights
 *  w_gate, w_up    [d_ff][D]      w_down [D][d_ff]
 *  state_out [n_slots][H_v][d_k][d_v] fp32 (M = S^T per value head)
 *  tail_out  NULL or [n_slots][C_tail][w-1] tail_dtype: the raw q | k | v
 *            projections of each live segment's last w-1 rows (zero before
 *            the segment's first row) */
typedef struct sr_block {
  const void* w_q;
  const void* w_k;
  const void* w_v;
  const void* w_z;
  const void* w_a;
  const void* w_b;
  const void* conv_w;
  const float* a_log;
  const float* dt_bias;
  const void* norm_o;
  const void* w_o;
  const void* ln_in;
  const void* ln_post;
  const void* w_gate;
  const void* w_up;
  const void* w_down;
  float* state_out;
  void* tail_out;
} sr_block;

/* Workspace bytes of sr_replay_group for t_total packed rows.  Host-only.
 * Supported shapes: anchor and weight dtype BF16, recurrence Gated DeltaNet,
 * d_k = d_v in {64, 128}, d_model a multiple of 256, d_ff a multiple of 128
 * (SR_ERR_BAD_SHAPE / SR_ERR_UNSUPPORTED_DTYPE otherwise). */
sr_status sr_group_workspace_size(const sr_shape* shape, int32_t d_ff, int64_t t_total, size_t* bytes);

/* Rebuilds the state (and conv tail) of every layer of one group for each
 * live segment of the batch.
 *  n_layers   1..64 blocks, in order
 *  anchors    [t_total][D] bf16: each segment's group-entry hidden states
 *  norm_eps   the RMSNorm epsilon (> 0)
 *  the varlen arguments, n_slots, varlen_status, workspace and stream as for
 *  sr_replay_state.  A segment of zero rows yields zero states and tails. */
sr_status sr_replay_group(const sr_shape* shape, int32_t d_ff, float norm_eps, int32_t n_layers,
                          const sr_block* blocks, const void* anchors, int32_t n_segments, int64_t t_total,
                          const int32_t* cu_seqlens, const int32_t* slot_ids, int32_t n_slots,
                          int32_t* varlen_status, void* workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SR_GROUP_H */
