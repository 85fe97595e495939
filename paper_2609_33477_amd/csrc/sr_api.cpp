// C ABI of the replay library: argument validation, workspace plan and the
// launch sequence per call.
//
// Every call first checks the device tables (one workgroup); every later
// kernel exits without writing if that check failed.
// bf16 / fp8 path, d_k = d_v, or d_k = 96, d_v = 192 with an even number of
// value heads (stream-ordered):
//   check          once per call, in the same launch the rows' position in
//                  their segment, rows left and slot (one block per segment)
//   proj_conv      per launch up to 4 layers: anchors x [W_k; W_v; W_a;
//                  W_b]^T fused with conv, SiLU, key norm and gates -> k_hat,
//                  v (bf16, head-major), log2 alpha, beta, the k | v part of
//                  the conv tail; blocks past the tiles compute its q part.
//                  96-wide key heads take 128 output columns each (zero
//                  pads) and land in a padded [H_k][T][128] key buffer; a
//                  192-wide value head lands as two padded halves, which
//                  the bf16 scan runs as two units of 128
// fp32 path, and 96 x 192 heads with an odd number of value heads, per layer:
//     proj_gemm    anchors x [W_k; W_v; W_a; W_b]^T -> P (fp32 workspace)
//     conv_gate    P -> k_hat, v, log alpha, beta, k | v tail
//     tail         q part of the conv tail (+ zeros before a segment's start)
// then one state launch per group of <= 32 layers writes the states (the
// pipelined bf16 scan, the fp32 scan, or the chunked kernel for the unfused
// 96 x 192 heads).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <vector>

#include "sr_internal.hpp"
#include "sr_replay.h"

namespace {

constexpr int64_t kAlign = 256;

int64_t align_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

int dtype_bytes(int dt) {
  switch (dt) {
    case SR_F32: return 4;
    case SR_BF16: return 2;
    case SR_FP8_E4M3: return 1;
  }
  return 0;
}

sr_status check_shape(const sr_shape* s) {
  if (!s) return SR_ERR_NULL_ARG;
  if (s->d_model < 64 || s->d_model > 16384 || s->d_model % 64 != 0) return SR_ERR_BAD_SHAPE;
  if (s->n_k_heads < 1 || s->n_v_heads < s->n_k_heads || s->n_v_heads > 128) return SR_ERR_BAD_SHAPE;
  if (s->n_v_heads % s->n_k_heads != 0) return SR_ERR_BAD_SHAPE;
  // square heads d_k = d_v in {32, 64, 128}, or OLMo-Hybrid's 96 x 192
  // (bf16 anchors, Gated DeltaNet only)
  const bool square = s->d_k == s->d_v && (s->d_k == 32 || s->d_k == 64 || s->d_k == 128);
  const bool rect = s->d_k == 96 && s->d_v == 192;
  if (!square && !rect) return SR_ERR_BAD_SHAPE;
  if (s->conv_width < 1 || s->conv_width > 4) return SR_ERR_BAD_SHAPE;
  if (!(s->l2_eps > 0.f)) return SR_ERR_BAD_SHAPE;
  const bool pair_ok = (s->anchor_dtype == SR_F32 && s->weight_dtype == SR_F32) ||
                       (s->anchor_dtype == SR_BF16 && s->weight_dtype == SR_BF16) ||
                       (s->anchor_dtype == SR_BF16 && s->weight_dtype == SR_FP8_E4M3);
  if (!pair_ok) return SR_ERR_UNSUPPORTED_DTYPE;
  if (s->conv_dtype != SR_F32 && s->conv_dtype != SR_BF16) return SR_ERR_UNSUPPORTED_DTYPE;
  if (s->tail_dtype != SR_F32 && s->tail_dtype != SR_BF16) return SR_ERR_UNSUPPORTED_DTYPE;
  if (s->recurrence != SR_RECURRENCE_GDN && s->recurrence != SR_RECURRENCE_DECAY) return SR_ERR_BAD_SHAPE;
  if (s->recurrence == SR_RECURRENCE_DECAY && s->anchor_dtype != SR_BF16) return SR_ERR_UNSUPPORTED_DTYPE;
  if (rect && (s->anchor_dtype != SR_BF16 || s->recurrence != SR_RECURRENCE_GDN)) return SR_ERR_UNSUPPORTED_DTYPE;
  return SR_OK;
}

struct Plan {
  int64_t ldp;                       // row pitch of P (floats)
  int64_t off_flag, off_p, off_info, off_k, off_v, off_g, off_b, total;
  int64_t k_stride, v_stride, g_stride;   // per-layer strides (elements)
  int op_dtype, op_bytes;
  bool fused;                        // bf16 anchors: projection fused with the conv epilogue
  bool rect;                         // fused rectangular heads: keys and value halves padded to 128 columns
  int k_pitch;                       // elements per K row
};

// Rectangular heads take the fused projection when their value columns fill
// whole 128-column wave blocks (the epilogue treats each block as one kind
// of column): an even number of 192-wide value heads.
bool rect_fused(const sr_shape* s) {
  return s->d_k == 96 && s->d_v == 192 && s->anchor_dtype == SR_BF16 &&
         ((int64_t)s->n_v_heads * s->d_v) % 128 == 0;
}

Plan make_plan(const sr_shape* s, int32_t n_layers, int64_t T) {
  Plan p{};
  const int64_t hk = s->n_k_heads, hv = s->n_v_heads;
  const int64_t N = hk * s->d_k + hv * s->d_v + 2 * hv;
  p.ldp = align_up(N, 4);
  p.op_dtype = s->anchor_dtype == SR_F32 ? SR_F32 : SR_BF16;
  p.op_bytes = dtype_bytes(p.op_dtype);
  p.rect = rect_fused(s);
  p.fused = p.op_dtype == SR_BF16 && (s->d_k == s->d_v || p.rect);
  p.k_pitch = p.rect ? 128 : s->d_k;
  p.k_stride = hk * T * p.k_pitch;
  p.v_stride = p.rect ? 2 * hv * T * p.k_pitch : hv * T * s->d_v;
  p.g_stride = hv * T;
  int64_t off = 0;
  p.off_flag = off; off = align_up(off + 4, kAlign);   // the table check's result word
  if (!p.fused) {                    // only the unfused paths store the projection
    p.off_p = off; off = align_up(off + T * p.ldp * 4, kAlign);
  } else {
    p.off_info = off; off = align_up(off + T * (int64_t)sizeof(sr::RowInfo), kAlign);
  }
  p.off_k = off; off = align_up(off + n_layers * p.k_stride * p.op_bytes, kAlign);
  p.off_v = off; off = align_up(off + n_layers * p.v_stride * p.op_bytes, kAlign);
  p.off_g = off; off = align_up(off + n_layers * p.g_stride * 4, kAlign);
  p.off_b = off; off = align_up(off + n_layers * p.g_stride * 4, kAlign);
  p.total = off;
  return p;
}

// ---- optional per-kernel event timing (benchmark instrumentation)
struct TimedLaunch {
  int kind;
  hipEvent_t start, stop;
};
bool g_timing = false;
uint32_t g_timing_kinds = ~0u;   // kinds bracketed by events while timing is on
std::vector<TimedLaunch> g_records;
std::vector<hipEvent_t> g_free_events;

hipEvent_t take_event() {
  if (!g_free_events.empty()) {
    hipEvent_t e = g_free_events.back();
    g_free_events.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// The HIP error and kernel of this thread's last failed launch.
thread_local hipError_t g_last_hip = hipSuccess;
thread_local int g_last_kind = -1;

hipError_t note(int kind, hipError_t e) {
  if (e != hipSuccess) {
    g_last_hip = e;
    g_last_kind = kind;
  }
  return e;
}

// Runs `launch` on stream s, bracketed by events when timing is enabled.
// The launchers report hipGetLastError(), which is per thread and sticky, so
// an error left by an earlier unrelated HIP call is cleared first.
template <typename F>
hipError_t timed(int kind, hipStream_t s, F&& launch) {
  (void)hipGetLastError();
  if (!g_timing || kind < 0 || kind >= 32 || !((g_timing_kinds >> kind) & 1u)) return note(kind, launch());
  TimedLaunch t{kind, take_event(), take_event()};
  if (!t.start || !t.stop) return note(kind, hipErrorOutOfMemory);
  hipError_t e = hipEventRecord(t.start, s);
  if (e != hipSuccess) return note(kind, e);
  e = launch();
  const hipError_t e2 = hipEventRecord(t.stop, s);
  if (e == hipSuccess && e2 != hipSuccess) return note(kind, e2);
  g_records.push_back(t);
  return note(kind, e);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

hipError_t sr::timed_launch(int kind, hipStream_t s, hipError_t (*launch)(void*), void* ctx) {
  return timed(kind, s, [&] { return launch(ctx); });
}

hipError_t sr::note_error(int kind, hipError_t e) { return note(kind, e); }

namespace {

sr_status check_layer(const sr_shape* s, const sr_layer& L, int64_t t_total) {
  if (t_total > 0 && !L.anchors) return SR_ERR_NULL_ARG;
  if (!L.w_k || !L.w_v || !L.w_a || !L.w_b || !L.conv_w || !L.a_log || !L.dt_bias || !L.state_out)
    return SR_ERR_NULL_ARG;
  if (s->weight_dtype == SR_FP8_E4M3) {
    if (!L.s_k || !L.s_v || !L.s_a || !L.s_b) return SR_ERR_NULL_ARG;
    if (L.w_q && !L.s_q) return SR_ERR_NULL_ARG;
  }
  const void* vec[] = {L.anchors, L.w_k, L.w_v, L.w_a, L.w_b, L.w_q, L.state_in, L.state_out};
  for (const void* p : vec)
    if (p && !aligned16(p)) return SR_ERR_MISALIGNED;
  return SR_OK;
}

}  // namespace

extern "C" {

size_t sr_state_bytes(const sr_shape* s) {
  if (!s) return 0;
  return (size_t)s->n_v_heads * (size_t)s->d_k * (size_t)s->d_v * 4u;
}

size_t sr_conv_tail_bytes(const sr_shape* s, int32_t with_q) {
  if (!s || s->conv_width < 1) return 0;
  const size_t c = (size_t)(with_q ? 2 : 1) * s->n_k_heads * s->d_k + (size_t)s->n_v_heads * s->d_v;
  return c * (size_t)(s->conv_width - 1) * (size_t)dtype_bytes(s->tail_dtype);
}

sr_status sr_replay_workspace_size(const sr_shape* shape, int32_t n_layers, int64_t t_total, size_t* bytes) {
  if (!bytes) return SR_ERR_NULL_ARG;
  const sr_status st = check_shape(shape);
  if (st != SR_OK) return st;
  if (n_layers < 1 || n_layers > 256 || t_total < 0 || t_total >= (int64_t(1) << 31)) return SR_ERR_BAD_SHAPE;
  *bytes = (size_t)make_plan(shape, n_layers, t_total).total;
  return SR_OK;
}

sr_status sr_replay_state(const sr_shape* shape, int32_t n_layers, const sr_layer* layers, int32_t n_segments,
                          int64_t t_total, const int32_t* cu_seqlens, const int32_t* slot_ids, int32_t n_slots,
                          int32_t* varlen_status, void* workspace, size_t workspace_bytes, void* stream) {
  sr_status st = check_shape(shape);
  if (st != SR_OK) return st;
  if (!layers) return SR_ERR_NULL_ARG;
  if (n_layers < 1 || n_layers > 256 || n_segments < 0 || t_total < 0 || t_total >= (int64_t(1) << 31))
    return SR_ERR_BAD_SHAPE;
  if (n_slots < 0 || n_slots > SR_MAX_SLOTS) return SR_ERR_BAD_SHAPE;
  if (n_segments == 0 && t_total != 0) return SR_ERR_BAD_SHAPE;
  if (n_segments > 0 && !cu_seqlens) return SR_ERR_NULL_ARG;
  for (int l = 0; l < n_layers; ++l) {
    st = check_layer(shape, layers[l], t_total);
    if (st != SR_OK) return st;
  }
  if (n_segments == 0) return SR_OK;     // nothing to replay, nothing written
  const Plan plan = make_plan(shape, n_layers, t_total);
  if ((size_t)plan.total > workspace_bytes) return SR_ERR_WORKSPACE_TOO_SMALL;
  if (!workspace) return SR_ERR_NULL_ARG;
  if ((reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) != 0) return SR_ERR_MISALIGNED;

  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  const int hk = shape->n_k_heads, hv = shape->n_v_heads, d = shape->d_k, w = shape->conv_width;
  const int c_k = hk * shape->d_k, c_v = hv * shape->d_v;
  const int c_kp = plan.rect ? hk * plan.k_pitch : c_k;   // key columns of the fused projection
  float* P = reinterpret_cast<float*>(ws + plan.off_p);
  char* Kb = ws + plan.off_k;
  char* Vb = ws + plan.off_v;
  float* Gb = reinterpret_cast<float*>(ws + plan.off_g);
  float* Bb = reinterpret_cast<float*>(ws + plan.off_b);

  int32_t* flag = reinterpret_cast<int32_t*>(ws + plan.off_flag);
  const bool fused = plan.fused;
  sr::RowInfo* info = reinterpret_cast<sr::RowInfo*>(ws + plan.off_info);
  // the table check, with the rows' segment info in the same launch when the
  // fused projection needs it
  if (timed(SR_KERNEL_VALIDATE, s, [&] {
        return fused && t_total > 0
                   ? sr::launch_validate_rows(cu_seqlens, slot_ids, n_segments, t_total, n_slots, flag,
                                              varlen_status, info, s)
                   : sr::launch_validate(cu_seqlens, slot_ids, n_segments, t_total, n_slots, flag, varlen_status, s);
      }) != hipSuccess)
    return SR_ERR_HIP;

  // fused projections are launched kProjBatch layers at a time
  sr::ProjConvBatch pb{};
  auto flush_proj = [&]() {
    if (pb.n_layers == 0) return hipSuccess;
    const hipError_t e = timed(SR_KERNEL_PROJ_CONV, s, [&] {
      return sr::launch_proj_conv(shape->weight_dtype, plan.rect ? plan.k_pitch : d, pb, s);
    });
    pb.n_layers = 0;
    return e;
  };
  for (int l = 0; l < n_layers; ++l) {
    const sr_layer& L = layers[l];
    const int c_q = L.w_q ? c_k : 0;
    const int c_tail = c_q + c_k + c_v;
    const sr::WeightSeg wseg[4] = {{L.w_k, L.s_k, 0, c_k},
                                   {L.w_v, L.s_v, c_k, c_k + c_v},
                                   {L.w_a, L.s_a, c_k + c_v, c_k + c_v + hv},
                                   {L.w_b, L.s_b, c_k + c_v + hv, c_k + c_v + 2 * hv}};
    const bool with_tail = L.tail_out && w > 1;
    sr::TailArgs t{};
    t.anchors = L.anchors;
    t.D = shape->d_model;
    t.w_q = L.w_q;
    t.s_q = L.s_q;
    t.c_q = c_q;
    t.cu = cu_seqlens;
    t.slot_ids = slot_ids;
    t.n_seg = n_segments;
    t.w = w;
    t.tail = L.tail_out;
    t.tail_bf16 = shape->tail_dtype == SR_BF16;
    t.c_tail = c_tail;
    t.err = flag;
    if (fused && (t_total > 0 || with_tail)) {
      // the q-tail blocks ride in the projection's grid (alone when T = 0)
      sr::ProjConvArgs f{};
      f.A = L.anchors;
      f.T = t_total;
      f.K = shape->d_model;
      f.N = c_kp + c_v + 2 * hv;
      f.n_wseg = 4;
      for (int i = 0; i < 4; ++i) f.seg[i] = wseg[i];
      f.info = info;
      f.conv_w = L.conv_w;
      f.conv_bf16 = shape->conv_dtype == SR_BF16;
      f.w = w;
      f.a_log = L.a_log;
      f.dt_bias = L.dt_bias;
      f.C_q = 0;
      f.C_k = c_kp;
      f.C_kv = c_kp + c_v;
      f.C_z = c_kp + c_v;
      f.k_real = plan.rect ? shape->d_k : 0;
      f.v_head = plan.rect ? shape->d_v : 0;
      f.q_scale = 1.f;
      f.H_v = hv;
      f.eps = shape->l2_eps;
      f.Kbuf = Kb + (int64_t)l * plan.k_stride * plan.op_bytes;
      f.Vbuf = Vb + (int64_t)l * plan.v_stride * plan.op_bytes;
      f.Gbuf = Gb + (int64_t)l * plan.g_stride;
      f.Bbuf = Bb + (int64_t)l * plan.g_stride;
      f.tail = w > 1 ? L.tail_out : nullptr;
      f.tail_bf16 = shape->tail_dtype == SR_BF16;
      f.c_tail = c_tail;
      f.tail_kv_off = c_q;
      f.err = flag;
      if (with_tail) {
        f.tq = t;
        f.tq_blocks = sr::tail_q_grid_x(t) * sr::tail_q_grid_y(t);
      }
      pb.layer[pb.n_layers] = f;
      pb.tq_off[pb.n_layers + 1] = pb.tq_off[pb.n_layers] + f.tq_blocks;
      if (++pb.n_layers == sr::kProjBatch && flush_proj() != hipSuccess) return SR_ERR_HIP;
    } else if (t_total > 0) {
      sr::GemmArgs g{};
      g.A = L.anchors;
      g.M = t_total;
      g.K = shape->d_model;
      g.N = c_k + c_v + 2 * hv;
      g.n_seg = 4;
      for (int i = 0; i < 4; ++i) g.seg[i] = wseg[i];
      g.C = P;
      g.ldc = plan.ldp;
      if (timed(SR_KERNEL_PROJ_GEMM, s, [&] { return sr::launch_proj_gemm(shape->anchor_dtype, shape->weight_dtype, g, s); }) != hipSuccess)
        return SR_ERR_HIP;

      sr::ConvGateArgs c{};
      c.P = P;
      c.ldp = plan.ldp;
      c.T = t_total;
      c.cu = cu_seqlens;
      c.slot_ids = slot_ids;
      c.n_seg = n_segments;
      c.conv_w = L.conv_w;
      c.w = w;
      c.a_log = L.a_log;
      c.dt_bias = L.dt_bias;
      c.H_k = hk;
      c.H_v = hv;
      c.d_k = shape->d_k;
      c.d_v = shape->d_v;
      c.eps = shape->l2_eps;
      c.Kbuf = Kb + (int64_t)l * plan.k_stride * plan.op_bytes;
      c.Vbuf = Vb + (int64_t)l * plan.v_stride * plan.op_bytes;
      c.Gbuf = Gb + (int64_t)l * plan.g_stride;
      c.Bbuf = Bb + (int64_t)l * plan.g_stride;
      c.tail = w > 1 ? L.tail_out : nullptr;
      c.c_tail = c_tail;
      c.tail_kv_off = c_q;
      c.err = flag;
      if (timed(SR_KERNEL_CONV_GATE, s, [&] { return sr::launch_conv_gate(plan.op_dtype, shape->conv_dtype, shape->tail_dtype, d, c, s); }) != hipSuccess)
        return SR_ERR_HIP;
    }
    if (with_tail && !fused) {
      if (timed(SR_KERNEL_TAIL, s, [&] { return sr::launch_tail(shape->anchor_dtype, shape->weight_dtype, shape->tail_dtype, t, s); }) != hipSuccess)
        return SR_ERR_HIP;
    }
  }

  if (flush_proj() != hipSuccess) return SR_ERR_HIP;

  for (int l0 = 0; l0 < n_layers; l0 += sr::kScanMaxLayers) {
    const int nl = n_layers - l0 < sr::kScanMaxLayers ? n_layers - l0 : sr::kScanMaxLayers;
    sr::ScanArgs a{};
    a.Kbuf = Kb + (int64_t)l0 * plan.k_stride * plan.op_bytes;
    a.Vbuf = Vb + (int64_t)l0 * plan.v_stride * plan.op_bytes;
    a.Gbuf = Gb + (int64_t)l0 * plan.g_stride;
    a.Bbuf = Bb + (int64_t)l0 * plan.g_stride;
    a.k_layer_stride = plan.k_stride;
    a.v_layer_stride = plan.v_stride;
    a.g_layer_stride = plan.g_stride;
    a.T = t_total;
    a.cu = cu_seqlens;
    a.slot_ids = slot_ids;
    a.n_seg = n_segments;
    a.H_k = hk;
    a.H_v = hv;
    a.n_layers = nl;
    a.err = flag;
    a.k_pitch = plan.k_pitch;
    for (int i = 0; i < nl; ++i) {
      a.state_in[i] = layers[l0 + i].state_in;
      a.state_out[i] = layers[l0 + i].state_out;
    }
    if (plan.rect) {
      // each value head as two square units of 128 (96 live rows and columns)
      a.H_v = 2 * hv;
      a.v_split = 2;
      a.st_rows = shape->d_k;
      a.st_cols = shape->d_v / 2;
      a.st_pitch = shape->d_v;
    }
    if (shape->recurrence == SR_RECURRENCE_DECAY) {
      if (timed(SR_KERNEL_DECAY_STATE, s, [&] { return sr::launch_decay_state(d, a, s); }) != hipSuccess)
        return SR_ERR_HIP;
    } else if (plan.rect) {
      if (timed(SR_KERNEL_GDN_SCAN, s, [&] { return sr::launch_scan(plan.op_dtype, plan.k_pitch, a, s); }) != hipSuccess)
        return SR_ERR_HIP;
    } else if (shape->d_k != shape->d_v) {
      if (timed(SR_KERNEL_GDN_SCAN, s, [&] { return sr::launch_chunk_state(shape->d_k, shape->d_v, a, s); }) != hipSuccess)
        return SR_ERR_HIP;
    } else if (timed(SR_KERNEL_GDN_SCAN, s, [&] { return sr::launch_scan(plan.op_dtype, d, a, s); }) != hipSuccess)
      return SR_ERR_HIP;
  }
  return SR_OK;
}

sr_status sr_kernel_timing_enable(int32_t enable) {
  g_timing = enable != 0;
  return SR_OK;
}

sr_status sr_kernel_timing_kinds(uint32_t mask) {
  g_timing_kinds = mask;
  return SR_OK;
}

sr_status sr_kernel_timing_read(double* ms, int64_t* launches) {
  if (!ms || !launches) return SR_ERR_NULL_ARG;
  for (int k = 0; k < SR_KERNEL_KINDS; ++k) {
    ms[k] = 0.0;
    launches[k] = 0;
  }
  sr_status st = SR_OK;
  for (TimedLaunch& t : g_records) {
    float el = 0.f;
    if (hipEventSynchronize(t.stop) != hipSuccess || hipEventElapsedTime(&el, t.start, t.stop) != hipSuccess) {
      st = SR_ERR_HIP;
    } else {
      ms[t.kind] += el;
      launches[t.kind] += 1;
    }
    g_free_events.push_back(t.start);
    g_free_events.push_back(t.stop);
  }
  g_records.clear();
  return st;
}

sr_status sr_last_hip_error(int32_t* hip_error, int32_t* kernel_kind, const char** message) {
  if (hip_error) *hip_error = (int32_t)g_last_hip;
  if (kernel_kind) *kernel_kind = g_last_kind;
  if (message) *message = hipGetErrorString(g_last_hip);
  return SR_OK;
}

const char* sr_status_str(sr_status status) {
  switch (status) {
    case SR_OK: return "ok";
    case SR_ERR_NULL_ARG: return "a required pointer is NULL";
    case SR_ERR_BAD_SHAPE: return "a size is outside the supported range";
    case SR_ERR_UNSUPPORTED_DTYPE: return "unsupported dtype or dtype combination";
    case SR_ERR_WORKSPACE_TOO_SMALL: return "workspace smaller than sr_replay_workspace_size()";
    case SR_ERR_MISALIGNED: return "a tensor pointer is not 16-byte aligned (workspace: 256-byte)";
    case SR_ERR_HIP: return "a HIP launch failed";
  }
  return "unknown status";
}

}  // extern "C"
