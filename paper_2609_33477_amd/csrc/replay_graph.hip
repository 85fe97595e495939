// Graph-bucketed, pipelined replay (Section 5.2: "Pipelined Anchor Fetching
// and Replay", "Layer-wise handoff", "Batched replay"; Section 6, "Replay
// graphs").
//
// One object serves one group of layers.  A captured graph freezes every
// pointer and size, so the object owns what a replay reads: per-layer anchor
// buffers of T_max rows and the padded segment table; the workspace is one
// region sized for the largest bucket, shared by every bucket's graph (runs on
// one object are stream-ordered), owned by the object or lent by the caller
// (several objects replayed in order on one stream can share one).
//
// Every bucket of B rows is captured at creation, so the hit path never
// captures.  A bucket's graph runs sr_replay_state over B rows and
// max_segments + 1 segments of the object's padded table.  A run picks the
// smallest bucket holding t_total, pads the caller's live table (n segments,
// t_total rows) into the object's table with one small kernel on the stream
// -- live segments as given, then one sentinel segment (slot -1) over rows
// t_total .. B - 1, then empty sentinels -- and launches that bucket's
// graph.  A batch no bucket holds (too many rows or
// segments) runs eagerly: on the object's buffers and workspace when they are
// large enough, otherwise on anchors and a workspace the caller passes.
// Padding rows are projected like any other row (their anchors are whatever
// the buffers hold; they start zeroed) and never reach a state: their
// segment's slot is -1.
//
// Anchor fetch: sr_replay_graph_fetch copies host ranges (pinned memory, the
// host anchor pool) into the object's buffers on a copy stream, after the
// object's previous run has finished reading them, and records a "ready"
// event that the next run waits for on its own stream; so the fetch of one
// group overlaps the replay of another.  Every run records a "done" event,
// which sr_replay_graph_wait hands to a consumer stream (the layer-wise
// handoff: the forward stream waits only where it needs this group's states).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

#include "sr_internal.hpp"
#include "sr_replay.h"
#include "sr_replay_graph.h"

namespace {

constexpr int kPadThreads = 256;

// Pads the caller's live table (cu [n + 1], slot [n] or null for identity)
// to max_seg + 1 segments over `rows` rows: live segments as given, then the
// sentinel over the rest of the rows, then empty sentinels.  It runs on the
// stream just before the bucket's graph, which reads the padded table from
// the object's own buffers.
__global__ __launch_bounds__(kPadThreads) void pad_table_kernel(const int32_t* __restrict__ cu,
                                                               const int32_t* __restrict__ slot, int32_t n,
                                                               int32_t* __restrict__ cu_pad,
                                                               int32_t* __restrict__ slot_pad, int32_t max_seg,
                                                               int32_t rows) {
  for (int s = threadIdx.x; s <= max_seg + 1; s += kPadThreads) {
    cu_pad[s] = s == 0 ? 0 : (s <= n ? cu[s] : rows);
    if (s <= max_seg) slot_pad[s] = s < n ? (slot ? slot[s] : s) : -1;
  }
}

}  // namespace

struct sr_replay_graph {
  sr_shape shape;
  int32_t n_layers = 0, max_seg = 0, n_slots = 0;
  int32_t* varlen_status = nullptr;      // caller's device word for the table check, or null
  int64_t t_max = 0;
  size_t row_bytes = 0;
  std::vector<sr_layer> layers;          // anchors replaced by the owned buffers
  std::vector<void*> anchor_buf;
  int32_t* cu_pad = nullptr;             // [max_seg + 2]
  int32_t* slot_pad = nullptr;           // [max_seg + 1]
  void* ws = nullptr;                    // shared by every bucket
  size_t ws_bytes = 0;
  bool own_ws = false;
  struct Bucket {
    int64_t rows;
    hipGraphExec_t exec = nullptr;
  };
  std::vector<Bucket> buckets;
  hipStream_t capture_stream = nullptr;
  hipEvent_t ready = nullptr;            // last fetch complete
  hipEvent_t done = nullptr;             // last run complete
  bool fetch_pending = false, ran = false;
};

namespace {

sr_status hip_fail(hipError_t e) {
  sr::note_error(SR_KERNEL_GRAPH, e);
  return SR_ERR_HIP;
}

void release(sr_replay_graph* g) {
  if (!g) return;
  for (auto& b : g->buckets)
    if (b.exec) (void)hipGraphExecDestroy(b.exec);
  for (void* p : g->anchor_buf)
    if (p) (void)hipFree(p);
  for (void* p : {(void*)g->cu_pad, (void*)g->slot_pad})
    if (p) (void)hipFree(p);
  if (g->own_ws && g->ws) (void)hipFree(g->ws);
  if (g->ready) (void)hipEventDestroy(g->ready);
  if (g->done) (void)hipEventDestroy(g->done);
  if (g->capture_stream) (void)hipStreamDestroy(g->capture_stream);
  delete g;
}

int elem_bytes(int dt) { return dt == SR_F32 ? 4 : (dt == SR_BF16 ? 2 : 1); }

// Captures bucket b: the replay over b.rows rows of the padded table.
sr_status capture(sr_replay_graph* g, sr_replay_graph::Bucket& b) {
  hipStream_t s = g->capture_stream;
  hipError_t e = hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal);
  if (e != hipSuccess) return hip_fail(e);
  const sr_status st = sr_replay_state(&g->shape, g->n_layers, g->layers.data(), g->max_seg + 1, b.rows, g->cu_pad,
                                       g->slot_pad, g->n_slots, g->varlen_status, g->ws, g->ws_bytes, s);
  hipGraph_t graph = nullptr;
  const hipError_t ee = hipStreamEndCapture(s, &graph);
  if (st != SR_OK || ee != hipSuccess || !graph) {
    if (graph) (void)hipGraphDestroy(graph);
    if (st != SR_OK) return st;
    return hip_fail(ee != hipSuccess ? ee : hipErrorUnknown);
  }
  const hipError_t ie = hipGraphInstantiate(&b.exec, graph, nullptr, nullptr, 0);
  (void)hipGraphDestroy(graph);
  return ie == hipSuccess ? SR_OK : hip_fail(ie);
}

}  // namespace

extern "C" {

sr_status sr_replay_graph_create(const sr_shape* shape, int32_t n_layers, const sr_layer* layers,
                                 int32_t n_slots, int32_t* varlen_status, int32_t max_segments,
                                 const int64_t* bucket_rows, int32_t n_buckets, void* workspace,
                                 size_t workspace_bytes, sr_replay_graph** out) {
  if (!shape || !layers || !bucket_rows || !out) return SR_ERR_NULL_ARG;
  *out = nullptr;
  if (n_layers < 1 || n_layers > 256 || max_segments < 1 || max_segments > 65536 || n_buckets < 1 || n_buckets > 64)
    return SR_ERR_BAD_SHAPE;
  if (n_slots < 0 || n_slots > SR_MAX_SLOTS) return SR_ERR_BAD_SHAPE;
  for (int i = 0; i < n_buckets; ++i)
    if (bucket_rows[i] < 1 || bucket_rows[i] > (int64_t)1 << 24 || (i > 0 && bucket_rows[i] <= bucket_rows[i - 1]))
      return SR_ERR_BAD_SHAPE;   // ascending, positive
  size_t need = 0;
  const sr_status ss = sr_replay_workspace_size(shape, n_layers, bucket_rows[n_buckets - 1], &need);
  if (ss != SR_OK) return ss;
  if (workspace) {
    if (workspace_bytes < need) return SR_ERR_WORKSPACE_TOO_SMALL;
    if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0) return SR_ERR_MISALIGNED;
  }
  auto* g = new sr_replay_graph();
  g->shape = *shape;
  g->n_layers = n_layers;
  g->max_seg = max_segments;
  g->n_slots = n_slots;
  g->varlen_status = varlen_status;
  g->t_max = bucket_rows[n_buckets - 1];
  g->row_bytes = (size_t)shape->d_model * elem_bytes(shape->anchor_dtype);
  hipError_t e = hipStreamCreateWithFlags(&g->capture_stream, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&g->ready, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&g->done, hipEventDisableTiming);
  g->layers.assign(layers, layers + n_layers);
  g->anchor_buf.assign(n_layers, nullptr);
  for (int l = 0; e == hipSuccess && l < n_layers; ++l) {
    e = hipMalloc(&g->anchor_buf[l], (size_t)g->t_max * g->row_bytes);
    if (e == hipSuccess) e = hipMemset(g->anchor_buf[l], 0, (size_t)g->t_max * g->row_bytes);
    g->layers[l].anchors = g->anchor_buf[l];
  }
  if (e == hipSuccess) e = hipMalloc((void**)&g->cu_pad, (max_segments + 2) * sizeof(int32_t));
  if (e == hipSuccess) e = hipMalloc((void**)&g->slot_pad, (max_segments + 1) * sizeof(int32_t));
  if (e == hipSuccess) {
    if (workspace) {
      g->ws = workspace;
      g->ws_bytes = workspace_bytes;
    } else {
      g->own_ws = true;
      g->ws_bytes = need > 0 ? need : 256;
      e = hipMalloc(&g->ws, g->ws_bytes);
    }
  }
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    release(g);
    return hip_fail(e);
  }
  // every bucket is captured now, so a run never captures
  for (int i = 0; i < n_buckets; ++i) {
    sr_replay_graph::Bucket b;
    b.rows = bucket_rows[i];
    g->buckets.push_back(b);
    const sr_status st = capture(g, g->buckets.back());
    if (st != SR_OK) {
      release(g);
      return st;
    }
  }
  // the capture stream is not used again: give its hardware queue back
  (void)hipStreamDestroy(g->capture_stream);
  g->capture_stream = nullptr;
  *out = g;
  return SR_OK;
}

void* sr_replay_graph_anchors(sr_replay_graph* g, int32_t layer) {
  if (!g || layer < 0 || layer >= g->n_layers) return nullptr;
  return g->anchor_buf[layer];
}

int64_t sr_replay_graph_max_rows(const sr_replay_graph* g) { return g ? g->t_max : 0; }

sr_status sr_replay_graph_fetch(sr_replay_graph* g, const sr_host_range* ranges, int32_t n_ranges,
                                void* copy_stream) {
  if (!g) return SR_ERR_NULL_ARG;
  if (n_ranges < 0 || (n_ranges > 0 && !ranges)) return n_ranges < 0 ? SR_ERR_BAD_SHAPE : SR_ERR_NULL_ARG;
  for (int i = 0; i < n_ranges; ++i) {
    const sr_host_range& r = ranges[i];
    if (r.layer < 0 || r.layer >= g->n_layers || r.dst_row < 0 || r.rows < 0 || r.dst_row + r.rows > g->t_max)
      return SR_ERR_BAD_SHAPE;
    if (r.rows > 0 && !r.src) return SR_ERR_NULL_ARG;
  }
  hipStream_t cs = (hipStream_t)copy_stream;
  // the previous run must have finished reading the buffers
  hipError_t e = g->ran ? hipStreamWaitEvent(cs, g->done, 0) : hipSuccess;
  for (int i = 0; e == hipSuccess && i < n_ranges; ++i) {
    const sr_host_range& r = ranges[i];
    if (r.rows == 0) continue;
    char* dst = static_cast<char*>(g->anchor_buf[r.layer]) + (size_t)r.dst_row * g->row_bytes;
    e = hipMemcpyAsync(dst, r.src, (size_t)r.rows * g->row_bytes, hipMemcpyHostToDevice, cs);
  }
  if (e == hipSuccess) e = hipEventRecord(g->ready, cs);
  if (e != hipSuccess) return hip_fail(e);
  g->fetch_pending = true;
  return SR_OK;
}

sr_status sr_replay_graph_run(sr_replay_graph* g, int32_t n_segments, int64_t t_total, const int32_t* cu_seqlens,
                              const int32_t* slot_ids, const void* const* eager_anchors, void* eager_workspace,
                              size_t eager_workspace_bytes, void* stream, int32_t* used_bucket) {
  if (!g) return SR_ERR_NULL_ARG;
  if (used_bucket) *used_bucket = -1;
  if (n_segments < 0 || t_total < 0) return SR_ERR_BAD_SHAPE;
  if (n_segments > 0 && !cu_seqlens) return SR_ERR_NULL_ARG;
  hipStream_t s = (hipStream_t)stream;
  const bool fits = t_total <= g->t_max && n_segments <= g->max_seg;
  // eager batches: checked in full before anything is enqueued
  std::vector<sr_layer> eager;
  void* ews = g->ws;
  size_t ews_bytes = g->ws_bytes;
  if (!fits) {
    eager = g->layers;
    if (t_total > g->t_max) {
      if (!eager_anchors) return SR_ERR_BAD_SHAPE;   // the owned buffers cannot hold the batch
      for (int l = 0; l < g->n_layers; ++l) eager[l].anchors = eager_anchors[l];
    }
    size_t need = 0;
    const sr_status st = sr_replay_workspace_size(&g->shape, g->n_layers, t_total, &need);
    if (st != SR_OK) return st;
    if (need > ews_bytes) {
      if (!eager_workspace || eager_workspace_bytes < need) return SR_ERR_WORKSPACE_TOO_SMALL;
      ews = eager_workspace;
      ews_bytes = eager_workspace_bytes;
    }
  }
  hipError_t e = g->fetch_pending ? hipStreamWaitEvent(s, g->ready, 0) : hipSuccess;
  if (e != hipSuccess) return hip_fail(e);
  g->fetch_pending = false;
  if (!fits) {
    const sr_status st = sr_replay_state(&g->shape, g->n_layers, eager.data(), n_segments, t_total, cu_seqlens,
                                         slot_ids, g->n_slots, g->varlen_status, ews, ews_bytes, stream);
    if (st != SR_OK) return st;
  } else {
    size_t bi = 0;
    while (g->buckets[bi].rows < t_total) ++bi;
    (void)hipGetLastError();
    hipLaunchKernelGGL(pad_table_kernel, dim3(1), dim3(kPadThreads), 0, s, cu_seqlens, slot_ids, n_segments, g->cu_pad,
                       g->slot_pad, g->max_seg, (int32_t)g->buckets[bi].rows);
    e = hipGetLastError();
    if (e == hipSuccess) e = hipGraphLaunch(g->buckets[bi].exec, s);
    if (e != hipSuccess) return hip_fail(e);
    if (used_bucket) *used_bucket = (int32_t)bi;
  }
  e = hipEventRecord(g->done, s);
  if (e != hipSuccess) return hip_fail(e);
  g->ran = true;
  return SR_OK;
}

sr_status sr_replay_graph_wait(sr_replay_graph* g, void* stream) {
  if (!g) return SR_ERR_NULL_ARG;
  if (!g->ran) return SR_OK;
  const hipError_t e = hipStreamWaitEvent((hipStream_t)stream, g->done, 0);
  return e == hipSuccess ? SR_OK : hip_fail(e);
}

sr_status sr_replay_graph_destroy(sr_replay_graph* g) {
  if (!g) return SR_OK;
  (void)hipDeviceSynchronize();
  release(g);
  return SR_OK;
}

}  // extern "C"
