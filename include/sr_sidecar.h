/*
 * sr_sidecar.h -- C ABI of the anchor sidecar's write and read paths
 * (hand-written HIP for gfx950 / MI355X), part of libsr_replay.
 *
 * Anchors are the retained input hidden states that replay consumes.  They
 * are kept at a fraction rho of token positions aligned to KV pages of p
 * tokens; the dense layout keeps the last p*rho rows of every page, so a token
 * at position t of its request is anchor (t mod p) - (p - p*rho) of page t / p
 * when t mod p >= p - p*rho (Section 4.2).  Every KV page owns one anchor
 * block holding its p*rho anchors for all A anchored layers (Section 5.1); the
 * pool of blocks is one device array laid out
 *     pool[n_blocks][n_layers][per_page][d]
 * and sidecar row r = block * per_page + slot names anchor `slot` of `block`.
 *
 * Write path (Section 5.1): the host builds, per serving step, a destination
 * row for every token of the step (sr_anchor_dest_table; -1 where nothing is
 * written, the paper's scratch address); during prefill the sampled tokens
 * are compacted on the device (sr_anchor_compact); an indexed copy then
 * writes each anchored layer's hidden row of those tokens into their blocks
 * (sr_anchor_write).
 *
 * Read path (Section 5.2): on a hit, replay needs only the last k anchors
 * before the matched boundary; sr_anchor_gather copies them out of the blocks
 * of the request's pages into the packed varlen batch that sr_replay_state()
 * consumes, request after request, and writes the segment offsets.
 *
 * Conventions are those of sr_replay.h: device pointers are owned by the
 * caller, nothing is allocated, work is only enqueued on `stream` (a
 * hipStream_t, NULL = default) and may be captured into a HIP graph (no
 * memset nodes are recorded), argument errors are reported before any launch
 * with nothing written, SR_ERR_HIP means a launch failed.  Rows are copied as
 * raw bytes, so any element type of elem_bytes bytes works.
 */
#ifndef SR_SIDECAR_H
#define SR_SIDECAR_H

#include <stddef.h>
#include <stdint.h>

#include "sr_replay.h"

#ifdef __cplusplus
extern "C" {
#endif

/* The block pool (Section 5.1).
 *  pool        device, [n_blocks][n_layers][per_page][d], 16-byte aligned
 *  n_blocks    >= 1
 *  n_layers    A, anchored layers per block, 1..64
 *  per_page    anchors per KV page (p * rho; 4 for p = 64, rho = 1/16), 1..64
 *  d           row width in elements; d * elem_bytes a multiple of 16
 *  elem_bytes  2 (bf16) or 4 (fp32) */
typedef struct sr_sidecar {
  void*   pool;
  int64_t n_blocks;
  int32_t n_layers;
  int32_t per_page;
  int32_t d;
  int32_t elem_bytes;
} sr_sidecar;

/* HOST function (all pointers are host memory; no device work): the
 * destination table of one serving step (Section 5.1) under the dense layout
 * (Section 4.2).
 *  positions   [n_tokens] position of token i in its request (>= 0)
 *  token_req   [n_tokens] request of token i, in [0, n_req)
 *  page_table  [page_cu[n_req]] anchor block of each page, request after
 *              request (page q of request r at page_cu[r] + q); -1 = the page
 *              has no block (nothing is written for its tokens)
 *  page_cu     [n_req + 1] offsets into page_table, non-decreasing from 0
 *  page_size   p >= 1;  per_page in 1..page_size
 *  dest        [n_tokens] out: block * per_page + slot for a sampled token
 *              whose page has a block, else -1
 * SR_ERR_BAD_SHAPE (nothing written) for a token whose request or position
 * is out of range; a position past the request's page table yields -1. */
sr_status sr_anchor_dest_table(const int32_t* positions, const int32_t* token_req, int32_t n_tokens,
                               const int32_t* page_table, const int32_t* page_cu, int32_t n_req,
                               int32_t page_size, int32_t per_page, int32_t* dest);

/* Device: stable compaction of the tokens that have a destination (the
 * prefill compaction of Section 5.1).
 *  dest     device [n_tokens]
 *  sel      device out [n_tokens]: the indices i with dest[i] >= 0, ascending,
 *           in sel[0 .. *n_sel - 1]; the rest of sel is not written
 *  n_sel    device out, one int32
 * One workgroup walks the table 8192 entries at a time (n_tokens <= 2^30). */
sr_status sr_anchor_compact(const int32_t* dest, int32_t n_tokens, int32_t* sel, int32_t* n_sel,
                            void* stream);

/* Device: the indexed copy of Section 5.1.  For every token i in the work
 * list, hidden[l] row i goes to layer l's copy of sidecar row dest[i]
 * (pool[dest[i] / per_page][l][dest[i] % per_page]), for l < sc->n_layers.
 *  hidden   HOST array of sc->n_layers device pointers, each [n_tokens][d]
 *           with sc->elem_bytes elements, 16-byte aligned
 *  dest     device [n_tokens]; rows < 0 are skipped; rows >= n_blocks *
 *           per_page are a precondition violation (not checked on device)
 *  sel      device work list from sr_anchor_compact (then n_sel is the device
 *           count), or NULL: every token, those with dest < 0 skipped (decode)
 * Two tokens with the same destination race (one of them wins). */
sr_status sr_anchor_write(const sr_sidecar* sc, const void* const* hidden, int32_t n_tokens,
                          const int32_t* dest, const int32_t* sel, const int32_t* n_sel, void* stream);

/* Device: the read path of Section 5.2.  Request r replays anchors
 * anchor_first[r] .. anchor_first[r] + n_anchors[r] - 1 of its anchor
 * sequence; anchor j of the sequence lives in block
 * block_table[block_cu[r] + j / per_page], slot j % per_page.  For each
 * requested layer layers[o], row cu_seqlens[r] + i of out[o] receives anchor
 * anchor_first[r] + i of request r.
 *  block_table  device [block_cu[n_req]] block ids (< n_blocks)
 *  block_cu     device [n_req + 1] offsets into block_table
 *  anchor_first, n_anchors   device [n_req], >= 0; the anchors must lie in
 *               the request's blocks (not checked on device)
 *  layers       HOST [n_out] layer indices in [0, n_layers), n_out 1..64
 *  out          HOST array of n_out device pointers, each [t_cap][d],
 *               16-byte aligned (NULL allowed when t_cap is 0)
 *  t_cap        rows available in each out[o]; rows past it are not written
 *  cu_seqlens   device out [n_req + 1]: prefix sums of n_anchors from 0 (the
 *               segment offsets sr_replay_state() takes)
 * n_req 0..65536. */
sr_status sr_anchor_gather(const sr_sidecar* sc, int32_t n_req, const int32_t* block_table,
                           const int32_t* block_cu, const int32_t* anchor_first, const int32_t* n_anchors,
                           const int32_t* layers, int32_t n_out, void* const* out, int64_t t_cap,
                           int32_t* cu_seqlens, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SR_SIDECAR_H */
