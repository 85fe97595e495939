/*
 * sr_replay_graph.h -- graph-bucketed replay (part of libsr_replay).
 *
 * The serving system batches cache hits into one varlen replay and captures
 * it into device graphs keyed by the batch's total packed length, padding a
 * batch up to its bucket with sentinel segments and falling back to eager
 * execution for batches no bucket holds (Section 5.2, "Batched replay").
 * A captured graph freezes its pointers and sizes, so this object owns what a
 * replay reads: one anchor buffer per layer of T_max = the largest bucket
 * rows, the segment table, and one workspace per bucket.  The caller writes
 * the anchors of a batch into sr_replay_graph_anchors(g, l) (rows
 * 0 .. t_total - 1, packed as for sr_replay_state) and calls
 * sr_replay_graph_run with its segment table; the states and tails go to the
 * layers' state_out / tail_out given at creation (frozen into the graphs),
 * exactly as sr_replay_state would write them.  A bucket's graph is captured
 * on its first use; a run writes the caller's table pointers and segment
 * count into a device parameter block (one one-thread kernel) and launches
 * it.  The caller's cu_seqlens / slot_ids must stay valid until the
 * launch has run.  Calls on one object must be ordered on one stream.
 */
#ifndef SR_REPLAY_GRAPH_H
#define SR_REPLAY_GRAPH_H

#include <stdint.h>

#include "sr_replay.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct sr_replay_graph sr_replay_graph;

/* Allocates the object (device memory: the anchor buffers, zeroed; the tables;
 * one workspace per bucket).  `layers` as for sr_replay_state, except that
 * `anchors` is ignored; their weight, state and tail pointers are used for
 * every run.  bucket_rows: n_buckets (1..64) strictly ascending row counts,
 * the last is T_max (<= 2^24).  max_segments: 1..65536 live segments per
 * graph run.  SR_ERR_HIP if an allocation fails (nothing is kept). */
sr_status sr_replay_graph_create(const sr_shape* shape, int32_t n_layers, const sr_layer* layers,
                                 int32_t max_segments, const int64_t* bucket_rows, int32_t n_buckets,
                                 sr_replay_graph** out);

/* Device buffer [T_max][d_model] of layer `layer`'s anchors, or NULL. */
void* sr_replay_graph_anchors(sr_replay_graph* g, int32_t layer);

/* T_max, the rows one run can hold (0 for NULL). */
int64_t sr_replay_graph_max_rows(const sr_replay_graph* g);

/* Replays a batch of n_segments segments over t_total <= T_max rows:
 * cu_seqlens / slot_ids are device arrays as for sr_replay_state (slot_ids may
 * be NULL: identity).  With n_segments <= max_segments it launches the graph of
 * the smallest bucket holding t_total rows (capturing it first if needed) on
 * `stream`; otherwise it runs sr_replay_state eagerly.  *used_bucket (if not
 * NULL) receives the bucket index, or -1 for the eager path. */
sr_status sr_replay_graph_run(sr_replay_graph* g, int32_t n_segments, int64_t t_total, const int32_t* cu_seqlens,
                              const int32_t* slot_ids, void* stream, int32_t* used_bucket);

/* Waits for the device, then frees everything. */
sr_status sr_replay_graph_destroy(sr_replay_graph* g);

#ifdef __cplusplus
}
#endif

#endif /* SR_REPLAY_GRAPH_H */
