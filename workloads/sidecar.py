"""Seeded synthetic inputs for the anchor sidecar's write and read paths.

Shared by the oracle-based tests and the HIP path, and holding none of the
method's arithmetic: it draws page tables (a random permutation of pool
blocks, as a paged allocator hands them out), token positions, raw element
bits for hidden states and pool contents, and replay requests.  Elements are
raw bit patterns (uint16 for bf16 rows, uint32 for fp32 rows): the sidecar
copies bytes, so both sides compare bits.

Defaults follow Section 4.2 and 5.1: 64-token pages with p * rho = 4 anchors
each, and for the Qwen3.5-4B shape A = 7 anchored layers of d = 2560 (Appendix
A, Eq. ours-bpt).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Sequence

import numpy as np

PAGE = 64
PER_PAGE = 4


def _bits(rng: np.random.Generator, shape, elem_bytes: int) -> np.ndarray:
    if elem_bytes == 2:
        return rng.integers(0, 1 << 16, shape, dtype=np.uint16)
    return rng.integers(0, 1 << 32, shape, dtype=np.uint32)


@dataclass
class WriteCase:
    """One serving step's tokens and the sidecar they write into."""
    positions: np.ndarray       # [n_tokens] int32
    token_req: np.ndarray       # [n_tokens] int32
    page_table: np.ndarray      # [page_cu[-1]] int32 (-1: no block)
    page_cu: np.ndarray         # [n_req + 1] int32
    hidden: List[np.ndarray]    # n_layers x [n_tokens][d] raw bits
    pool: np.ndarray            # [n_blocks * n_layers * PER_PAGE][d] raw bits (initial contents)
    n_layers: int
    n_blocks: int

    def page_tables(self) -> List[List[int]]:
        return [list(map(int, self.page_table[self.page_cu[r]:self.page_cu[r + 1]]))
                for r in range(len(self.page_cu) - 1)]


def write_case(seed: int, spans: Sequence[tuple], n_layers: int, d: int, elem_bytes: int = 2,
               hole_frac: float = 0.0) -> WriteCase:
    """A step whose request r covers positions spans[r] = (start, stop): a
    prefill chunk (start 0), a later chunk, or a decode token (stop = start +
    1).  Each request owns ceil(stop / 64) pages; a fraction hole_frac of the
    pages has no block."""
    rng = np.random.default_rng((seed, 1))
    pages = [(stop + PAGE - 1) // PAGE for _, stop in spans]
    n_blocks = max(1, sum(pages))
    perm = rng.permutation(n_blocks).astype(np.int32)
    table = perm[:sum(pages)].copy()
    if hole_frac > 0 and table.size:
        table[rng.random(table.size) < hole_frac] = -1
    page_cu = np.concatenate([[0], np.cumsum(pages)]).astype(np.int32)
    positions = np.concatenate([np.arange(a, b) for a, b in spans] or [np.zeros(0)]).astype(np.int32)
    token_req = np.concatenate([np.full(b - a, r) for r, (a, b) in enumerate(spans)]
                               or [np.zeros(0)]).astype(np.int32)
    hidden = [_bits(rng, (len(positions), d), elem_bytes) for _ in range(n_layers)]
    pool = _bits(rng, (n_blocks * n_layers * PER_PAGE, d), elem_bytes)
    return WriteCase(positions, token_req, table, page_cu, hidden, pool, n_layers, n_blocks)


@dataclass
class GatherCase:
    """Replay requests over a filled pool: request r has n_total[r] anchors
    in its pages and replays the last n_anchors[r] of them."""
    pool: np.ndarray            # [n_blocks * n_layers * PER_PAGE][d] raw bits
    block_table: np.ndarray     # [block_cu[-1]] int32
    block_cu: np.ndarray        # [n_req + 1] int32
    anchor_first: np.ndarray    # [n_req] int32
    n_anchors: np.ndarray       # [n_req] int32
    n_layers: int
    n_blocks: int

    def block_tables(self) -> List[List[int]]:
        return [list(map(int, self.block_table[self.block_cu[r]:self.block_cu[r + 1]]))
                for r in range(len(self.block_cu) - 1)]


def gather_case(seed: int, ks: Sequence[int], n_layers: int, d: int, elem_bytes: int = 2,
                max_extra: int = 9) -> GatherCase:
    """Request r replays ks[r] anchors that end a history of ks[r] + e
    anchors, e drawn from 0..max_extra, so replay starts anywhere in a page."""
    rng = np.random.default_rng((seed, 2))
    extra = rng.integers(0, max_extra + 1, len(ks))
    n_total = [int(k) + int(e) for k, e in zip(ks, extra)]
    pages = [(n + PER_PAGE - 1) // PER_PAGE for n in n_total]
    n_blocks = max(1, sum(pages))
    table = rng.permutation(n_blocks).astype(np.int32)[:sum(pages)]
    block_cu = np.concatenate([[0], np.cumsum(pages)]).astype(np.int32)
    pool = _bits(rng, (n_blocks * n_layers * PER_PAGE, d), elem_bytes)
    first = np.array([n - int(k) for n, k in zip(n_total, ks)], dtype=np.int32)
    return GatherCase(pool, table, block_cu, first, np.asarray(ks, dtype=np.int32), n_layers, n_blocks)
