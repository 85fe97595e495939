// Graph-bucketed replay (Section 5.2, "Batched replay"; the serving system
// captures replay into graphs keyed by the batch's total packed length).
//
// A graph freezes every pointer and size it was captured with, so the object
// owns the buffers a replay reads: per-layer anchor buffers of T_max rows,
// the padded segment table, and one workspace per bucket.  A bucket of
// B rows is one captured graph that
//   1. pads the live table (n segments, t_total rows) to max_segments + 1
//      segments covering exactly B rows:
//      live segments as given, then one sentinel segment (slot -1) over rows
//      t_total .. B - 1, then empty sentinel segments;
//   2. runs sr_replay_state over B rows and max_segments + 1 segments.
// A call writes the caller's table pointers and live segment count into a
// device parameter block (one one-thread kernel) and launches the smallest
// bucket that holds t_total; a batch with more segments than
// max_segments runs eagerly on the largest bucket's workspace.  Padding rows are
// projected like any other row (their anchors are whatever the buffers hold;
// they start zeroed) and never reach a state: their segment's slot is -1.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

#include "sr_internal.hpp"
#include "sr_replay.h"
#include "sr_replay_graph.h"

namespace {

constexpr int kPadThreads = 256;

// The batch a graph launch replays: the caller's table and its live segment
// count, written by a one-thread kernel before each launch.
struct PadParams {
  const int32_t* cu;     // [n + 1], cu[n] = live rows
  const int32_t* slot;   // [n] or null (identity)
  int32_t n;
};

__global__ void set_params_kernel(PadParams* p, const int32_t* cu, const int32_t* slot, int32_t n) {
  p->cu = cu;
  p->slot = slot;
  p->n = n;
}

// Pads the live table to max_seg + 1 segments over `rows` rows: live
// segments as given, then the sentinel over the rest of the rows, then empty
// sentinels.
__global__ __launch_bounds__(kPadThreads) void pad_table_kernel(const PadParams* __restrict__ p,
                                                               int32_t* __restrict__ cu_pad,
                                                               int32_t* __restrict__ slot_pad, int32_t max_seg,
                                                               int32_t rows) {
  const int n = p->n;
  const int32_t* cu = p->cu;
  const int32_t* slot = p->slot;
  for (int s = threadIdx.x; s <= max_seg + 1; s += kPadThreads) {
    cu_pad[s] = s == 0 ? 0 : (s <= n ? cu[s] : rows);
    if (s <= max_seg) slot_pad[s] = s < n ? (slot ? slot[s] : s) : -1;
  }
}

}  // namespace

struct sr_replay_graph {
  sr_shape shape;
  int32_t n_layers = 0, max_seg = 0;
  int64_t t_max = 0;
  int device = 0;
  std::vector<sr_layer> layers;          // anchors replaced by the owned buffers
  std::vector<void*> anchor_buf;
  PadParams* params = nullptr;
  int32_t* cu_pad = nullptr;             // [max_seg + 2]
  int32_t* slot_pad = nullptr;           // [max_seg + 1]
  struct Bucket {
    int64_t rows;
    void* ws = nullptr;
    size_t ws_bytes = 0;
    hipGraphExec_t exec = nullptr;
  };
  std::vector<Bucket> buckets;
  hipStream_t capture_stream = nullptr;
};

namespace {

void release(sr_replay_graph* g) {
  if (!g) return;
  for (auto& b : g->buckets) {
    if (b.exec) (void)hipGraphExecDestroy(b.exec);
    if (b.ws) (void)hipFree(b.ws);
  }
  for (void* p : g->anchor_buf)
    if (p) (void)hipFree(p);
  for (void* p : {(void*)g->params, (void*)g->cu_pad, (void*)g->slot_pad})
    if (p) (void)hipFree(p);
  if (g->capture_stream) (void)hipStreamDestroy(g->capture_stream);
  delete g;
}

int elem_bytes(int dt) { return dt == SR_F32 ? 4 : (dt == SR_BF16 ? 2 : 1); }

// Captures bucket b: the padding kernel and the replay over b.rows rows.
sr_status capture(sr_replay_graph* g, sr_replay_graph::Bucket& b) {
  hipStream_t s = g->capture_stream;
  if (hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal) != hipSuccess) return SR_ERR_HIP;
  hipLaunchKernelGGL(pad_table_kernel, dim3(1), dim3(kPadThreads), 0, s, g->params, g->cu_pad, g->slot_pad,
                     g->max_seg, (int32_t)b.rows);
  const hipError_t le = hipGetLastError();
  const sr_status st = le == hipSuccess
                           ? sr_replay_state(&g->shape, g->n_layers, g->layers.data(), g->max_seg + 1, b.rows,
                                             g->cu_pad, g->slot_pad, b.ws, b.ws_bytes, s)
                           : SR_ERR_HIP;
  hipGraph_t graph = nullptr;
  const hipError_t ee = hipStreamEndCapture(s, &graph);
  if (st != SR_OK || ee != hipSuccess || !graph) {
    if (graph) (void)hipGraphDestroy(graph);
    return st != SR_OK ? st : SR_ERR_HIP;
  }
  const hipError_t ie = hipGraphInstantiate(&b.exec, graph, nullptr, nullptr, 0);
  (void)hipGraphDestroy(graph);
  return ie == hipSuccess ? SR_OK : SR_ERR_HIP;
}

}  // namespace

extern "C" {

sr_status sr_replay_graph_create(const sr_shape* shape, int32_t n_layers, const sr_layer* layers,
                                 int32_t max_segments, const int64_t* bucket_rows, int32_t n_buckets,
                                 sr_replay_graph** out) {
  if (!shape || !layers || !bucket_rows || !out) return SR_ERR_NULL_ARG;
  *out = nullptr;
  if (n_layers < 1 || max_segments < 1 || max_segments > 65536 || n_buckets < 1 || n_buckets > 64)
    return SR_ERR_BAD_SHAPE;
  for (int i = 0; i < n_buckets; ++i)
    if (bucket_rows[i] < 1 || bucket_rows[i] > (int64_t)1 << 24 || (i > 0 && bucket_rows[i] <= bucket_rows[i - 1]))
      return SR_ERR_BAD_SHAPE;   // ascending, positive
  size_t probe = 0;
  const sr_status ss = sr_replay_workspace_size(shape, n_layers, bucket_rows[n_buckets - 1], &probe);
  if (ss != SR_OK) return ss;
  auto* g = new sr_replay_graph();
  g->shape = *shape;
  g->n_layers = n_layers;
  g->max_seg = max_segments;
  g->t_max = bucket_rows[n_buckets - 1];
  if (hipGetDevice(&g->device) != hipSuccess) {
    release(g);
    return SR_ERR_HIP;
  }
  const size_t row_bytes = (size_t)shape->d_model * elem_bytes(shape->anchor_dtype);
  bool ok = hipStreamCreateWithFlags(&g->capture_stream, hipStreamNonBlocking) == hipSuccess;
  g->layers.assign(layers, layers + n_layers);
  g->anchor_buf.assign(n_layers, nullptr);
  for (int l = 0; ok && l < n_layers; ++l) {
    ok = hipMalloc(&g->anchor_buf[l], (size_t)g->t_max * row_bytes) == hipSuccess &&
         hipMemset(g->anchor_buf[l], 0, (size_t)g->t_max * row_bytes) == hipSuccess;
    g->layers[l].anchors = g->anchor_buf[l];
  }
  ok = ok && hipMalloc((void**)&g->params, sizeof(PadParams)) == hipSuccess &&
       hipMalloc((void**)&g->cu_pad, (max_segments + 2) * sizeof(int32_t)) == hipSuccess &&
       hipMalloc((void**)&g->slot_pad, (max_segments + 1) * sizeof(int32_t)) == hipSuccess;
  for (int i = 0; ok && i < n_buckets; ++i) {
    sr_replay_graph::Bucket b;
    b.rows = bucket_rows[i];
    ok = sr_replay_workspace_size(shape, n_layers, b.rows, &b.ws_bytes) == SR_OK &&
         hipMalloc(&b.ws, b.ws_bytes > 0 ? b.ws_bytes : 256) == hipSuccess;
    g->buckets.push_back(b);
  }
  ok = ok && hipDeviceSynchronize() == hipSuccess;
  if (!ok) {
    release(g);
    return SR_ERR_HIP;
  }
  *out = g;
  return SR_OK;
}

void* sr_replay_graph_anchors(sr_replay_graph* g, int32_t layer) {
  if (!g || layer < 0 || layer >= g->n_layers) return nullptr;
  return g->anchor_buf[layer];
}

int64_t sr_replay_graph_max_rows(const sr_replay_graph* g) { return g ? g->t_max : 0; }

sr_status sr_replay_graph_run(sr_replay_graph* g, int32_t n_segments, int64_t t_total, const int32_t* cu_seqlens,
                              const int32_t* slot_ids, void* stream, int32_t* used_bucket) {
  if (!g) return SR_ERR_NULL_ARG;
  if (used_bucket) *used_bucket = -1;
  if (n_segments < 0 || t_total < 0 || t_total > g->t_max) return SR_ERR_BAD_SHAPE;
  if (n_segments > 0 && !cu_seqlens) return SR_ERR_NULL_ARG;
  hipStream_t s = (hipStream_t)stream;
  if (n_segments > g->max_seg) {
    // eager: the caller's table as given, the largest bucket's workspace
    auto& b = g->buckets.back();
    return sr_replay_state(&g->shape, g->n_layers, g->layers.data(), n_segments, t_total, cu_seqlens, slot_ids,
                           b.ws, b.ws_bytes, stream);
  }
  size_t bi = 0;
  while (g->buckets[bi].rows < t_total) ++bi;
  auto& b = g->buckets[bi];
  if (!b.exec) {
    const sr_status st = capture(g, b);
    if (st != SR_OK) return st;
  }
  (void)hipGetLastError();
  hipLaunchKernelGGL(set_params_kernel, dim3(1), dim3(1), 0, s, g->params, cu_seqlens, slot_ids, n_segments);
  if (hipGetLastError() != hipSuccess) return SR_ERR_HIP;
  if (hipGraphLaunch(b.exec, s) != hipSuccess) return SR_ERR_HIP;
  if (used_bucket) *used_bucket = (int32_t)bi;
  return SR_OK;
}

sr_status sr_replay_graph_destroy(sr_replay_graph* g) {
  if (!g) return SR_OK;
  (void)hipDeviceSynchronize();
  release(g);
  return SR_OK;
}

}  // extern "C"
