/*
 * sr_replay_graph.h -- graph-bucketed, pipelined replay (part of libsr_replay).
 *
 * The serving system fetches a hit's anchors from its host pinned pool on a
 * dedicated copy stream, replays the linear-attention groups in order on a
 * replay stream, and lets the forward stream wait only where it first reads a
 * group's rebuilt states (Section 5.2, "Pipelined Anchor Fetching and
 * Replay", "Layer-wise handoff").  Replay runs from graphs captured once at
 * initialisation, one per total-packed-length bucket, with batches padded up
 * to their bucket by sentinel segments; a batch no bucket holds is replayed
 * eagerly (Section 5.2, "Batched replay" and the fail-closed paragraph;
 * Section 6, "Replay graphs").
 *
 * One sr_replay_graph serves one group of layers.  A captured graph freezes
 * its pointers and sizes, so the object owns the anchor buffers a replay reads
 * (one per layer, T_max = the largest bucket rows, zeroed at creation) and the
 * padded segment table.  The workspace is one region sized for the largest
 * bucket and shared by all of the object's graphs; the caller may lend it
 * (several objects replayed in order on one stream can share one region).
 * The states and tails go to the layers' state_out / tail_out given at
 * creation, exactly as sr_replay_state would write them.  The caller's weight,
 * state and tail buffers must outlive the object.
 *
 * Ordering: runs of one object must be ordered on one stream, and its fetches
 * on one copy stream.  sr_replay_graph_fetch waits (on the copy stream) for
 * the object's previous run before overwriting its buffers and records an
 * event that the next run waits for (on its stream); the caller's host memory
 * must stay valid until the copy has run, and must be pinned (hipHostMalloc)
 * for the copy to overlap other work.
 */
#ifndef SR_REPLAY_GRAPH_H
#define SR_REPLAY_GRAPH_H

#include <stddef.h>
#include <stdint.h>

#include "sr_replay.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct sr_replay_graph sr_replay_graph;

/* One host range of anchor rows for sr_replay_graph_fetch: `rows` rows of
 * d_model elements (anchor_dtype) at `src`, copied into layer `layer`'s
 * buffer starting at row `dst_row`. */
typedef struct sr_host_range {
  const void* src;
  int32_t layer;
  int64_t dst_row;
  int64_t rows;
} sr_host_range;

/* Allocates the object and captures the graph of every bucket (device
 * memory: the anchor buffers, zeroed; the tables; the workspace unless lent).
 * `layers` as for sr_replay_state, except that `anchors` is ignored; their
 * weight, state and tail pointers are frozen into the graphs, and so are
 * n_slots (the slot count of every layer's state_out / tail_out) and
 * varlen_status (NULL or a device word receiving each run's table check, as
 * for sr_replay_state; the check covers the padded table, so a live table
 * whose rows overrun its bucket is refused on the device).
 * bucket_rows: n_buckets (1..64) strictly ascending row counts, the last is
 * T_max (<= 2^24).  max_segments: 1..65536 live segments per graph run.
 * workspace: NULL (the object allocates its own) or a device region of
 * workspace_bytes >= sr_replay_workspace_size(shape, n_layers, T_max),
 * 256-byte aligned, that the caller keeps alive and uses for nothing else
 * while the object's runs are in flight.
 * SR_ERR_HIP (details in sr_last_hip_error) if an allocation or capture
 * fails; nothing is kept then. */
sr_status sr_replay_graph_create(const sr_shape* shape, int32_t n_layers, const sr_layer* layers,
                                 int32_t n_slots, int32_t* varlen_status, int32_t max_segments,
                                 const int64_t* bucket_rows, int32_t n_buckets, void* workspace,
                                 size_t workspace_bytes, sr_replay_graph** out);

/* Device buffer [T_max][d_model] of layer `layer`'s anchors, or NULL. */
void* sr_replay_graph_anchors(sr_replay_graph* g, int32_t layer);

/* T_max, the rows one graph run can hold (0 for NULL). */
int64_t sr_replay_graph_max_rows(const sr_replay_graph* g);

/* Enqueues host -> device copies of `n_ranges` ranges into the object's
 * anchor buffers on `copy_stream` (hipStream_t), after the object's last run
 * has finished reading them, and records the event the next run waits for.
 * SR_ERR_BAD_SHAPE (nothing enqueued) if a range leaves its buffer or names
 * no layer of the object. */
sr_status sr_replay_graph_fetch(sr_replay_graph* g, const sr_host_range* ranges, int32_t n_ranges,
                                void* copy_stream);

/* Replays a batch of n_segments segments over t_total rows on `stream`, after
 * the object's last fetch: cu_seqlens / slot_ids are device arrays as for
 * sr_replay_state (slot_ids may be NULL: identity; both must stay valid until
 * the launch has run).
 *  - t_total <= T_max and n_segments <= max_segments: launches the captured
 *    graph of the smallest bucket holding t_total rows (anchors: the object's
 *    buffers).
 *  - Otherwise an eager sr_replay_state call.  With t_total > T_max its
 *    anchors are eager_anchors[l] (host array of n_layers device pointers,
 *    [t_total][d_model] each; NULL gives SR_ERR_BAD_SHAPE); otherwise the
 *    object's buffers.  Its workspace is the object's when large enough,
 *    else eager_workspace (eager_workspace_bytes >=
 *    sr_replay_workspace_size(...t_total), else SR_ERR_WORKSPACE_TOO_SMALL).
 * Every check runs before anything is enqueued.  *used_bucket (if not NULL)
 * receives the bucket index, or -1 for the eager path. */
sr_status sr_replay_graph_run(sr_replay_graph* g, int32_t n_segments, int64_t t_total, const int32_t* cu_seqlens,
                              const int32_t* slot_ids, const void* const* eager_anchors, void* eager_workspace,
                              size_t eager_workspace_bytes, void* stream, int32_t* used_bucket);

/* Makes `stream` wait (on the device, not the host) until the object's last
 * run has finished: the hand-off to the first consumer of this group's
 * states.  A no-op before the first run. */
sr_status sr_replay_graph_wait(sr_replay_graph* g, void* stream);

/* Waits for the device, then frees everything the object owns. */
sr_status sr_replay_graph_destroy(sr_replay_graph* g);

#ifdef __cplusplus
}
#endif

#endif /* SR_REPLAY_GRAPH_H */
