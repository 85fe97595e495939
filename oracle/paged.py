"""Oracle for the anchor sidecar's write and read paths (plain numpy, byte copies).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle``: only the test suite,
``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg use it, and
it shares no code with the HIP path.

What it computes:

* Section 4.2 (token-wise sparse anchors, dense layout): anchors are kept at a
  fraction rho of positions, aligned to KV pages of p tokens; the dense layout
  keeps the last p*rho rows of every page.  A token at position t of its
  request is an anchor iff t mod p >= p - p*rho, and it is anchor number
  (t mod p) - (p - p*rho) of page t // p.
* Section 5.1 (anchor sidecar): each KV page owns one anchor block holding its
  p*rho anchors for every anchored layer; a block is laid out here as
  [layer][anchor in page][d] (for Qwen3.5-4B: 7 layers x 4 anchors x 2560 bf16
  = 143,360 bytes, the "about 140 KB" per page the paper quotes).
* Section 5.1 (writing anchors): the host precomputes, per serving step, a
  destination for every token of the step: the sidecar row of a sampled token
  whose page has a block, and "none" otherwise (the paper's scratch address,
  which the sidecar ignores; here -1).  During prefill the sampled tokens are
  compacted first; the indexed copy then writes each anchored layer's hidden
  state row of every sampled token to its block.
* Section 5.2 (pipelined anchor fetching): on a hit the replay reads only the
  last k anchors before the cached boundary, which lie in the blocks of the
  matched pages; they are gathered, request after request, into the packed
  varlen batch the replay consumes, with segment offsets cu_seqlens.

Sidecar row numbering: row r = block * per_page + slot addresses anchor
``slot`` of block ``block``; with n_layers anchored layers, layer l's copy of
that row sits at flat row (block * n_layers + l) * per_page + slot of the pool
viewed as [n_rows][d].
"""
from __future__ import annotations

from typing import Sequence, Tuple

import numpy as np


def block_bytes(n_layers: int, per_page: int, d: int, elem_bytes: int) -> int:
    """Bytes of one page's anchor block (Section 5.1)."""
    return n_layers * per_page * d * elem_bytes


def dense_anchor_slot(t: int, page_size: int, per_page: int) -> int:
    """Anchor number within its page of position t under the dense layout
    (Section 4.2), or -1 if t is not an anchor."""
    r = t % page_size
    first = page_size - per_page
    return r - first if r >= first else -1


def dest_table(positions: Sequence[int], token_req: Sequence[int], page_tables: Sequence[Sequence[int]],
               page_size: int, per_page: int) -> np.ndarray:
    """Per-token sidecar destination row for one serving step (Section 5.1).

    positions[i] is token i's position in its request token_req[i];
    page_tables[r][q] is the anchor block of page q of request r, or -1 where
    the page has none.  Returns int32 rows, -1 for tokens that are not written.
    """
    out = np.full(len(positions), -1, dtype=np.int32)
    for i, (t, r) in enumerate(zip(positions, token_req)):
        slot = dense_anchor_slot(int(t), page_size, per_page)
        if slot < 0:
            continue
        q = int(t) // page_size
        table = page_tables[int(r)]
        if q >= len(table) or table[q] < 0:
            continue
        out[i] = table[q] * per_page + slot
    return out


def compact(dest: np.ndarray) -> np.ndarray:
    """Indices of the tokens that have a destination, in token order (the
    prefill compaction before the indexed copy, Section 5.1)."""
    return np.array([i for i in range(len(dest)) if dest[i] >= 0], dtype=np.int32)


def anchor_write(pool: np.ndarray, hidden: Sequence[np.ndarray], dest: np.ndarray, per_page: int) -> np.ndarray:
    """The indexed copy (Section 5.1): a copy of ``pool`` ([n_rows][d]) where
    hidden[l][i] has been written to layer l's copy of sidecar row dest[i] for
    every token i with dest[i] >= 0.  Rows are copied as raw elements."""
    out = pool.copy()
    n_layers = len(hidden)
    for i in range(len(dest)):
        row = int(dest[i])
        if row < 0:
            continue
        block, slot = divmod(row, per_page)
        for l in range(n_layers):
            out[(block * n_layers + l) * per_page + slot] = hidden[l][i]
    return out


def anchor_gather(pool: np.ndarray, n_layers: int, per_page: int, block_tables: Sequence[Sequence[int]],
                  anchor_first: Sequence[int], n_anchors: Sequence[int],
                  layers: Sequence[int]) -> Tuple[np.ndarray, np.ndarray]:
    """The read path (Section 5.2): for request r, anchors anchor_first[r] ..
    anchor_first[r] + n_anchors[r] - 1 of its anchor sequence (anchor j lives
    in block block_tables[r][j // per_page], slot j % per_page), for each
    requested layer, packed request after request.

    Returns (out [len(layers)][T][d], cu_seqlens [n_req + 1] int32)."""
    cu = [0]
    for n in n_anchors:
        cu.append(cu[-1] + int(n))
    d = pool.shape[1]
    out = np.zeros((len(layers), cu[-1], d), dtype=pool.dtype)
    for r in range(len(n_anchors)):
        for j in range(int(n_anchors[r])):
            a = int(anchor_first[r]) + j
            block = int(block_tables[r][a // per_page])
            slot = a % per_page
            for li, l in enumerate(layers):
                out[li, cu[r] + j] = pool[(block * n_layers + l) * per_page + slot]
    return out, np.array(cu, dtype=np.int32)
