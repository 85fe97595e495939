"""Pins of the anchor sidecar oracle (oracle.paged) against facts fixed
outside it: the paper's per-token anchor bytes and per-page block size
(Appendix A, Eq. ours-bpt; Section 5.1), the anchor count of the dense layout
in closed form (Section 4.2), a library routine for the compaction, the
block layout read as a 4-D array, and brute-force selection of the sampled
rows by position.  Each test names the mistake it is there to catch."""
import json
import os

import numpy as np
import pytest

from oracle import paged

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_block_bytes_match_the_paper():
    """Catches a block that drops a layer or the per-page anchor count."""
    g = json.load(open(os.path.join(GOLDEN, "anchor_block_sizes.json")))
    p, rho, eb = g["page_size"], g["rho"], g["elem_bytes"]
    per_page = int(p * rho)
    assert per_page == 4
    for name, m in g["models"].items():
        blk = paged.block_bytes(m["A"], per_page, m["d"], eb)
        assert blk == m["bytes_per_token"] * p, name
        if "block_kb_approx" in m:
            assert abs(blk / 1024 - m["block_kb_approx"]) < 0.02 * m["block_kb_approx"]


@pytest.mark.parametrize("L", [0, 1, 59, 60, 61, 63, 64, 65, 124, 125, 128, 1000, 4096])
def test_dense_layout_anchor_count_closed_form(L):
    """A prefill of L tokens keeps 4 floor(L/64) + max(0, L mod 64 - 60)
    anchors (the last 4 rows of every page, Section 4.2), i.e. exactly rho L
    when L is a whole number of pages.  Catches an off-by-one page edge."""
    pages = (L + 63) // 64
    dest = paged.dest_table(range(L), [0] * L, [list(range(pages))], 64, 4)
    n = int((dest >= 0).sum())
    assert n == 4 * (L // 64) + max(0, L % 64 - 60)
    if L % 64 == 0:
        assert n == L // 16


def test_dense_slots_are_the_last_rows_of_each_page():
    """Positions 60..63 of a page are its anchors 0..3; nothing else is one."""
    slots = [paged.dense_anchor_slot(t, 64, 4) for t in range(192)]
    for t, s in enumerate(slots):
        assert s == (t % 64 - 60 if t % 64 >= 60 else -1)


def test_compact_matches_flatnonzero():
    """Catches an unstable or off-by-one compaction."""
    rng = np.random.default_rng(3)
    dest = np.where(rng.random(1000) < 0.1, rng.integers(0, 500, 1000), -1).astype(np.int32)
    assert np.array_equal(paged.compact(dest), np.flatnonzero(dest >= 0).astype(np.int32))
    assert paged.compact(np.full(5, -1, np.int32)).size == 0


def _prefill(rng, lens, n_layers, d, page_size=64, per_page=4, holes=()):
    """Hidden states of a prefill of several requests, their page tables (a
    random permutation of blocks, with some pages missing) and the tokens'
    positions and owners, packed request after request."""
    pages = [(L + page_size - 1) // page_size for L in lens]
    perm = rng.permutation(sum(pages))
    tables, o = [], 0
    for r, n in enumerate(pages):
        tables.append([int(b) for b in perm[o:o + n]])
        o += n
    for r, q in holes:
        tables[r][q] = -1
    positions = np.concatenate([np.arange(L) for L in lens]).astype(np.int32)
    owner = np.concatenate([np.full(L, r) for r, L in enumerate(lens)]).astype(np.int32)
    hidden = [rng.integers(0, 1 << 16, (len(positions), d), dtype=np.uint16) for _ in range(n_layers)]
    return tables, positions, owner, hidden, sum(pages)


def test_write_lays_blocks_out_layer_major_per_page():
    """After the indexed copy, the pool read as [block][layer][anchor][d]
    holds, at (page's block, l, t mod 64 - 60), layer l's hidden row of every
    sampled token t whose page has a block.  Catches swapped layer and slot
    strides, or a write to a missing page."""
    rng = np.random.default_rng(7)
    lens, A, d = [130, 64, 7, 250], 3, 16
    tables, pos, owner, hidden, n_blocks = _prefill(rng, lens, A, d, holes=[(3, 1)])
    dest = paged.dest_table(pos, owner, tables, 64, 4)
    pool0 = rng.integers(0, 1 << 16, (n_blocks * A * 4, d), dtype=np.uint16)
    pool = paged.anchor_write(pool0, hidden, dest, 4)
    p4, p04 = pool.reshape(n_blocks, A, 4, d), pool0.reshape(n_blocks, A, 4, d)
    touched = np.zeros((n_blocks, 4), bool)
    for i, (t, r) in enumerate(zip(pos, owner)):
        if t % 64 < 60:
            continue
        blk = tables[r][t // 64]
        if blk < 0:
            assert dest[i] == -1
            continue
        touched[blk, t % 64 - 60] = True
        for l in range(A):
            assert np.array_equal(p4[blk, l, t % 64 - 60], hidden[l][i])
    for b in range(n_blocks):
        for s in range(4):
            if not touched[b, s]:
                assert np.array_equal(p4[b, :, s], p04[b, :, s])


def test_gather_returns_the_last_k_anchors_in_position_order():
    """Write a prefill, then gather the last k anchors of each request: they
    are the hidden rows of that request's last k sampled positions, by brute
    force over positions.  Catches a wrong suffix start, a reversed page
    order, or a dropped request."""
    rng = np.random.default_rng(11)
    lens, A, d = [640, 200, 64, 1000], 4, 8
    tables, pos, owner, hidden, n_blocks = _prefill(rng, lens, A, d)
    dest = paged.dest_table(pos, owner, tables, 64, 4)
    pool = paged.anchor_write(np.zeros((n_blocks * A * 4, d), np.uint16), hidden, dest, 4)
    n_total = [4 * (L // 64) + max(0, L % 64 - 60) for L in lens]
    ks = [min(n, k) for n, k in zip(n_total, [17, 9, 4, 0])]
    first = [n - k for n, k in zip(n_total, ks)]
    layers = [2, 0]
    out, cu = paged.anchor_gather(pool, A, 4, tables, first, ks, layers)
    assert list(cu) == list(np.cumsum([0] + ks))
    for r in range(len(lens)):
        idx = [i for i in range(len(pos)) if owner[i] == r and pos[i] % 64 >= 60]
        want = idx[len(idx) - ks[r]:]
        for li, l in enumerate(layers):
            for j, i in enumerate(want):
                assert np.array_equal(out[li, cu[r] + j], hidden[l][i])
