// C ABI of group replay chaining (include/sr_group.h): host checks, the
// workspace plan and the launch sequence.
//
// Per call (stream-ordered):
//   validate (with the row info)        once
//   rmsnorm(anchors) -> x (bf16), h (fp32 residual stream)
//   per layer j < n - 1:
//     proj_conv   x -> q, k, v, z (bf16, head-major), log2 alpha, beta, conv tail
//     gdn_output  -> state_out, y = RMSNorm(o) * w * SiLU(z) (bf16 [T][H_v d])
//     gemm resid  h += y W_o^T
//     rmsnorm     h -> u
//     gemm swiglu m = SiLU(u W_gate^T) * (u W_up^T)
//     gemm resid  h += m W_down^T
//     rmsnorm     h -> x (the next layer's input, its ln_in)
//   last layer: the state-only path of sr_replay_state (projection without
//   q / z, with the q part of the tail in its grid; chunked scan).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "sr_group.h"
#include "sr_internal.hpp"
#include "sr_replay.h"

namespace {

constexpr int64_t kAlign = 256;
int64_t align_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

struct GroupPlan {
  int64_t off_flag, off_info, off_h, off_x, off_q, off_k, off_v, off_z, off_g, off_b, off_y, off_m, total;
};

GroupPlan make_group_plan(const sr_shape* s, int32_t d_ff, int64_t T) {
  GroupPlan p{};
  const int64_t D = s->d_model, hk = s->n_k_heads, hv = s->n_v_heads, d = s->d_k;
  int64_t off = 0;
  auto take = [&](int64_t bytes) {
    const int64_t o = off;
    off = align_up(off + bytes, kAlign);
    return o;
  };
  p.off_flag = take(4);
  p.off_info = take(T * (int64_t)sizeof(sr::RowInfo));
  p.off_h = take(T * D * 4);
  p.off_x = take(T * D * 2);                 // the mixer's input, then the MLP's
  p.off_q = take(hk * T * d * 2);
  p.off_k = take(hk * T * d * 2);
  p.off_v = take(hv * T * d * 2);
  p.off_z = take(hv * T * d * 2);
  p.off_g = take(hv * T * 4);
  p.off_b = take(hv * T * 4);
  p.off_y = take(T * hv * d * 2);
  // the MLP's hidden rows reuse q | k | v | z (dead once y is formed) when
  // they fit there
  const int64_t qkvz = p.off_g - p.off_q;
  p.off_m = T * d_ff * 2 <= qkvz ? p.off_q : take(T * d_ff * 2);
  p.total = off;
  return p;
}

sr_status check_group_shape(const sr_shape* s, int32_t d_ff) {
  size_t probe = 0;
  const sr_status st = sr_replay_workspace_size(s, 1, 0, &probe);   // the single-layer checks
  if (st != SR_OK) return st;
  if (s->anchor_dtype != SR_BF16 || s->weight_dtype != SR_BF16) return SR_ERR_UNSUPPORTED_DTYPE;
  if (s->recurrence != SR_RECURRENCE_GDN) return SR_ERR_UNSUPPORTED_DTYPE;
  if (s->d_k != 64 && s->d_k != 128) return SR_ERR_BAD_SHAPE;
  if (s->d_model % 256 != 0 || d_ff < 128 || d_ff % 128 != 0 || d_ff > (1 << 20)) return SR_ERR_BAD_SHAPE;
  return SR_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

sr_status check_block(const sr_block& b) {
  const void* req[] = {b.w_q, b.w_k, b.w_v, b.w_z, b.w_a, b.w_b, b.conv_w, b.a_log, b.dt_bias, b.norm_o,
                       b.w_o, b.ln_in, b.ln_post, b.w_gate, b.w_up, b.w_down, b.state_out};
  for (const void* p : req)
    if (!p) return SR_ERR_NULL_ARG;
  const void* vec[] = {b.w_q, b.w_k, b.w_v, b.w_z, b.w_a, b.w_b, b.w_o, b.ln_in, b.ln_post,
                       b.w_gate, b.w_up, b.w_down, b.state_out};
  for (const void* p : vec)
    if (!aligned16(p)) return SR_ERR_MISALIGNED;
  return SR_OK;
}

}  // namespace

extern "C" {

sr_status sr_group_workspace_size(const sr_shape* shape, int32_t d_ff, int64_t t_total, size_t* bytes) {
  if (!bytes) return SR_ERR_NULL_ARG;
  const sr_status st = check_group_shape(shape, d_ff);
  if (st != SR_OK) return st;
  if (t_total < 0 || t_total >= (int64_t(1) << 31)) return SR_ERR_BAD_SHAPE;
  *bytes = (size_t)make_group_plan(shape, d_ff, t_total).total;
  return SR_OK;
}

sr_status sr_replay_group(const sr_shape* shape, int32_t d_ff, float norm_eps, int32_t n_layers,
                          const sr_block* blocks, const void* anchors, int32_t n_segments, int64_t t_total,
                          const int32_t* cu_seqlens, const int32_t* slot_ids, int32_t n_slots,
                          int32_t* varlen_status, void* workspace, size_t workspace_bytes, void* stream) {
  sr_status st = check_group_shape(shape, d_ff);
  if (st != SR_OK) return st;
  if (!blocks) return SR_ERR_NULL_ARG;
  if (n_layers < 1 || n_layers > 64 || n_segments < 0 || t_total < 0 || t_total >= (int64_t(1) << 31))
    return SR_ERR_BAD_SHAPE;
  if (!(norm_eps > 0.f)) return SR_ERR_BAD_SHAPE;
  if (n_slots < 0 || n_slots > SR_MAX_SLOTS) return SR_ERR_BAD_SHAPE;
  if (n_segments == 0 && t_total != 0) return SR_ERR_BAD_SHAPE;
  if (n_segments > 0 && !cu_seqlens) return SR_ERR_NULL_ARG;
  if (t_total > 0 && !anchors) return SR_ERR_NULL_ARG;
  if (anchors && !aligned16(anchors)) return SR_ERR_MISALIGNED;
  for (int l = 0; l < n_layers; ++l) {
    st = check_block(blocks[l]);
    if (st != SR_OK) return st;
  }
  if (n_segments == 0) return SR_OK;
  const GroupPlan plan = make_group_plan(shape, d_ff, t_total);
  if ((size_t)plan.total > workspace_bytes) return SR_ERR_WORKSPACE_TOO_SMALL;
  if (!workspace) return SR_ERR_NULL_ARG;
  if ((reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) != 0) return SR_ERR_MISALIGNED;

  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  const int D = shape->d_model, hk = shape->n_k_heads, hv = shape->n_v_heads, d = shape->d_k;
  const int w = shape->conv_width;
  const int c_q = hk * d, c_k = 2 * hk * d, c_kv = 2 * hk * d + hv * d, c_z = c_kv + hv * d;
  const int c_tail = c_kv;                      // q | k | v
  const int64_t T = t_total;
  int32_t* flag = reinterpret_cast<int32_t*>(ws + plan.off_flag);
  sr::RowInfo* info = reinterpret_cast<sr::RowInfo*>(ws + plan.off_info);
  float* H = reinterpret_cast<float*>(ws + plan.off_h);
  void* X = ws + plan.off_x;
  void *Qb = ws + plan.off_q, *Kb = ws + plan.off_k, *Vb = ws + plan.off_v, *Zb = ws + plan.off_z;
  float* Gb = reinterpret_cast<float*>(ws + plan.off_g);
  float* Bb = reinterpret_cast<float*>(ws + plan.off_b);
  void* Y = ws + plan.off_y;
  void* Mh = ws + plan.off_m;
  auto fail = [&](hipError_t e) { return e == hipSuccess ? SR_OK : SR_ERR_HIP; };

  // the table check, with the rows' segment info for the fused projection
  // in the same launch when there are rows
  if (fail(sr::timed_call(SR_KERNEL_VALIDATE, s, [&] {
        return T > 0 ? sr::launch_validate_rows(cu_seqlens, slot_ids, n_segments, t_total, n_slots, flag,
                                                varlen_status, info, s)
                     : sr::launch_validate(cu_seqlens, slot_ids, n_segments, t_total, n_slots, flag, varlen_status, s);
      })) != SR_OK)
    return SR_ERR_HIP;
  if (T == 0) {
    // every segment is empty: zero states and tails, through the state-only
    // path (its own table check writes the same flag word)
    for (int l = 0; l < n_layers; ++l) {
      sr_layer L{};
      const sr_block& B = blocks[l];
      L.w_k = B.w_k; L.w_v = B.w_v; L.w_a = B.w_a; L.w_b = B.w_b; L.w_q = B.w_q;
      L.conv_w = B.conv_w; L.a_log = B.a_log; L.dt_bias = B.dt_bias;
      L.state_out = B.state_out; L.tail_out = B.tail_out;
      st = sr_replay_state(shape, 1, &L, n_segments, 0, cu_seqlens, slot_ids, n_slots, nullptr, workspace,
                           workspace_bytes, stream);
      if (st != SR_OK) return st;
    }
    return SR_OK;
  }

  auto rmsnorm = [&](const void* x, bool in_bf16, const void* wgt, void* out, float* copy) {
    sr::RmsNormArgs r{};
    r.x = x; r.in_bf16 = in_bf16; r.T = T; r.D = D; r.w = wgt; r.eps = norm_eps; r.out = out; r.copy = copy;
    r.err = flag;
    return sr::timed_call(SR_KERNEL_RMSNORM, s, [&] { return sr::launch_rmsnorm(r, s); });
  };
  auto gemm = [&](int mode, const void* A, int K, int N, const void* Bw, const void* B2, void* C, int64_t ldc) {
    sr::BlockGemmArgs g{};
    g.A = A; g.M = T; g.K = K; g.N = N; g.B = Bw; g.B2 = B2; g.C = C; g.ldc = ldc; g.err = flag;
    const int kind = mode == sr::kGemmSwiglu ? SR_KERNEL_GEMM_SWIGLU : SR_KERNEL_GEMM_RESID;
    return sr::timed_call(kind, s, [&] { return sr::launch_block_gemm(mode, g, s); });
  };

  if (fail(rmsnorm(anchors, true, blocks[0].ln_in, X, H)) != SR_OK) return SR_ERR_HIP;
  const size_t conv_eb = shape->conv_dtype == SR_BF16 ? 2 : 4;
  for (int l = 0; l < n_layers; ++l) {
    const sr_block& B = blocks[l];
    const bool last = l + 1 == n_layers;
    sr::ProjConvArgs f{};
    f.A = X;
    f.T = T;
    f.K = D;
    f.info = info;
    f.conv_bf16 = shape->conv_dtype == SR_BF16;
    f.w = w;
    f.a_log = B.a_log;
    f.dt_bias = B.dt_bias;
    f.H_v = hv;
    f.eps = shape->l2_eps;
    f.Kbuf = Kb;
    f.Vbuf = Vb;
    f.Gbuf = Gb;
    f.Bbuf = Bb;
    f.tail = w > 1 ? B.tail_out : nullptr;
    f.tail_bf16 = shape->tail_dtype == SR_BF16;
    f.c_tail = c_tail;
    f.err = flag;
    if (!last) {
      // q | k | v | z | a | b, q scaled by d^-1/2; the conv tail's channels are the columns
      f.N = c_z + 2 * hv;
      f.n_wseg = 6;
      f.seg[0] = {B.w_q, nullptr, 0, c_q};
      f.seg[1] = {B.w_k, nullptr, c_q, c_k};
      f.seg[2] = {B.w_v, nullptr, c_k, c_kv};
      f.seg[3] = {B.w_z, nullptr, c_kv, c_z};
      f.seg[4] = {B.w_a, nullptr, c_z, c_z + hv};
      f.seg[5] = {B.w_b, nullptr, c_z + hv, c_z + 2 * hv};
      f.conv_w = B.conv_w;
      f.C_q = c_q;
      f.C_k = c_k;
      f.C_kv = c_kv;
      f.C_z = c_z;
      f.q_scale = 1.f / __builtin_sqrtf((float)d);
      f.Qbuf = Qb;
      f.Zbuf = Zb;
      f.tail_kv_off = 0;
    } else {
      // state only: k | v | a | b (the q channels of the tail come from the q-tail blocks)
      f.N = c_kv - c_q + 2 * hv;
      f.n_wseg = 4;
      f.seg[0] = {B.w_k, nullptr, 0, c_k - c_q};
      f.seg[1] = {B.w_v, nullptr, c_k - c_q, c_kv - c_q};
      f.seg[2] = {B.w_a, nullptr, c_kv - c_q, c_kv - c_q + hv};
      f.seg[3] = {B.w_b, nullptr, c_kv - c_q + hv, c_kv - c_q + 2 * hv};
      f.conv_w = static_cast<const char*>(B.conv_w) + (size_t)c_q * w * conv_eb;
      f.C_q = 0;
      f.C_k = c_k - c_q;
      f.C_kv = c_kv - c_q;
      f.C_z = c_kv - c_q;
      f.q_scale = 1.f;
      f.tail_kv_off = c_q;
    }
    if (w > 1 && B.tail_out) {
      // blocks appended to the projection's grid: the q channels of the tail
      // (last layer) and the zeros at tail positions before each segment's
      // first row (the projection's epilogue writes the rows themselves)
      sr::TailArgs t{};
      t.anchors = X;
      t.D = D;
      t.w_q = last ? B.w_q : nullptr;
      t.c_q = last ? c_q : 0;
      t.cu = cu_seqlens;
      t.slot_ids = slot_ids;
      t.n_seg = n_segments;
      t.w = w;
      t.tail = B.tail_out;
      t.tail_bf16 = shape->tail_dtype == SR_BF16;
      t.c_tail = c_tail;
      t.err = flag;
      f.tq = t;
      f.tq_blocks = sr::tail_q_grid_x(t) * sr::tail_q_grid_y(t);
    }
    if (fail(sr::timed_call(SR_KERNEL_PROJ_CONV, s, [&] { return sr::launch_proj_conv(SR_BF16, d, f, s); })) !=
        SR_OK)
      return SR_ERR_HIP;

    if (!last) {
      sr::OutputArgs o{};
      o.Qbuf = Qb; o.Kbuf = Kb; o.Vbuf = Vb; o.Zbuf = Zb; o.Gbuf = Gb; o.Bbuf = Bb;
      o.T = T; o.cu = cu_seqlens; o.slot_ids = slot_ids; o.n_seg = n_segments; o.H_k = hk; o.H_v = hv;
      o.norm_w = B.norm_o; o.eps = norm_eps; o.Y = Y; o.state_out = B.state_out; o.err = flag;
      if (fail(sr::timed_call(SR_KERNEL_GDN_OUTPUT, s, [&] { return sr::launch_gdn_output(d, o, s); })) != SR_OK)
        return SR_ERR_HIP;
      if (fail(gemm(sr::kGemmResid, Y, hv * d, D, B.w_o, nullptr, H, D)) != SR_OK) return SR_ERR_HIP;
      if (fail(rmsnorm(H, false, B.ln_post, X, nullptr)) != SR_OK) return SR_ERR_HIP;
      if (fail(gemm(sr::kGemmSwiglu, X, D, 2 * d_ff, B.w_gate, B.w_up, Mh, d_ff)) != SR_OK) return SR_ERR_HIP;
      if (fail(gemm(sr::kGemmResid, Mh, d_ff, D, B.w_down, nullptr, H, D)) != SR_OK) return SR_ERR_HIP;
      if (fail(rmsnorm(H, false, blocks[l + 1].ln_in, X, nullptr)) != SR_OK) return SR_ERR_HIP;
    } else {
      sr::ScanArgs a{};
      a.Kbuf = Kb;
      a.Vbuf = Vb;
      a.Gbuf = Gb;
      a.Bbuf = Bb;
      a.k_layer_stride = (int64_t)hk * T * d;
      a.v_layer_stride = (int64_t)hv * T * d;
      a.g_layer_stride = (int64_t)hv * T;
      a.T = T;
      a.cu = cu_seqlens;
      a.slot_ids = slot_ids;
      a.n_seg = n_segments;
      a.H_k = hk;
      a.H_v = hv;
      a.n_layers = 1;
      a.err = flag;
      a.state_in[0] = nullptr;
      a.state_out[0] = B.state_out;
      if (fail(sr::timed_call(SR_KERNEL_GDN_SCAN, s, [&] { return sr::launch_scan(SR_BF16, d, a, s); })) != SR_OK)
        return SR_ERR_HIP;
    }
  }
  return SR_OK;
}

}  // extern "C"
