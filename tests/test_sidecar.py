"""Anchor sidecar write and read paths (Sections 4.2, 5.1, 5.2) against the
oracle (oracle.paged), bit for bit: these are byte copies and index work.

CPU tests: the host-side destination table (a host function of the C ABI)
and the host argument checks of the device entry points, which return before
any launch.  GPU tests: compaction, indexed copy and gather through the C ABI
on seeded cases with ragged and empty requests, holes in the page tables,
both row widths, a short output buffer, and the full Qwen3.5-4B-sized gather
of the 16-request workload."""
import ctypes

import numpy as np
import pytest

from oracle import paged
from workloads import sidecar as wsc

sr = pytest.importorskip("paper_2609_33477_amd.binding",
                         reason="libsr_replay.so not built (run __graft_entry__.build())")

SR_OK, SR_ERR_NULL_ARG, SR_ERR_BAD_SHAPE, SR_ERR_UNSUPPORTED_DTYPE, SR_ERR_MISALIGNED = 0, 1, 2, 3, 5


# ------------------------------------------------------------------- host
@pytest.mark.parametrize("seed,spans,holes", [
    (0, [(0, 1000), (0, 64), (0, 59)], 0.0),            # prefills, one with no anchor yet
    (1, [(0, 4096), (128, 700), (63, 64), (60, 61)], 0.2),  # later chunks and decode tokens, missing pages
    (2, [(5000, 5001)] * 1 + [(0, 300)], 0.5),
])
def test_dest_table_matches_oracle(seed, spans, holes):
    c = wsc.write_case(seed, spans, n_layers=1, d=8, hole_frac=holes)
    got = sr.anchor_dest_table(c.positions, c.token_req, c.page_table, c.page_cu, wsc.PAGE, wsc.PER_PAGE)
    want = paged.dest_table(c.positions, c.token_req, c.page_tables(), wsc.PAGE, wsc.PER_PAGE)
    assert np.array_equal(got, want)


def test_dest_table_position_past_the_page_table_is_skipped():
    got = sr.anchor_dest_table([61, 200], [0, 0], [5], [0, 1], 64, 4)
    assert list(got) == [5 * 4 + 1, -1]


def test_dest_table_rejects_bad_tokens():
    for pos, req in (([-1], [0]), ([3], [1]), ([3], [-1])):
        with pytest.raises(sr.SrError):
            sr.anchor_dest_table(pos, req, [0], [0, 1], 64, 4)
    with pytest.raises(sr.SrError):
        sr.anchor_dest_table([1], [0], [0], [0, 1], 64, 65)    # per_page > page_size


def _sidecar(pool=16, n_blocks=1, n_layers=1, per_page=4, d=8, eb=2):
    return sr.SrSidecar(pool, n_blocks, n_layers, per_page, d, eb)


def test_device_entry_points_reject_bad_arguments_before_any_launch():
    lib = sr.LIB
    one = (ctypes.c_void_p * 1)(16)
    lay = (ctypes.c_int32 * 1)(0)
    cases = [
        (lib.sr_anchor_write(None, one, 1, 16, None, None, None), SR_ERR_NULL_ARG),
        (lib.sr_anchor_write(ctypes.byref(_sidecar(pool=0)), one, 1, 16, None, None, None), SR_ERR_NULL_ARG),
        (lib.sr_anchor_write(ctypes.byref(_sidecar(n_layers=65)), one, 1, 16, None, None, None), SR_ERR_BAD_SHAPE),
        (lib.sr_anchor_write(ctypes.byref(_sidecar(eb=3)), one, 1, 16, None, None, None), SR_ERR_UNSUPPORTED_DTYPE),
        (lib.sr_anchor_write(ctypes.byref(_sidecar(d=7)), one, 1, 16, None, None, None), SR_ERR_BAD_SHAPE),
        (lib.sr_anchor_write(ctypes.byref(_sidecar(pool=8)), one, 1, 16, None, None, None), SR_ERR_MISALIGNED),
        (lib.sr_anchor_write(ctypes.byref(_sidecar()), (ctypes.c_void_p * 1)(8), 1, 16, None, None, None),
         SR_ERR_MISALIGNED),
        (lib.sr_anchor_write(ctypes.byref(_sidecar()), one, 1, 16, 16, None, None), SR_ERR_NULL_ARG),
        (lib.sr_anchor_write(ctypes.byref(_sidecar()), one, -1, 16, None, None, None), SR_ERR_BAD_SHAPE),
        (lib.sr_anchor_write(ctypes.byref(_sidecar()), one, 0, None, None, None, None), SR_OK),
        (lib.sr_anchor_compact(16, -1, 16, 16, None), SR_ERR_BAD_SHAPE),
        (lib.sr_anchor_compact(16, 4, 16, None, None), SR_ERR_NULL_ARG),
        (lib.sr_anchor_gather(ctypes.byref(_sidecar()), 1, 16, 16, 16, 16, (ctypes.c_int32 * 1)(1), 1, one, 4,
                              16, None), SR_ERR_BAD_SHAPE),
        (lib.sr_anchor_gather(ctypes.byref(_sidecar()), 1, 16, 16, 16, 16, lay, 0, one, 4, 16, None),
         SR_ERR_BAD_SHAPE),
        (lib.sr_anchor_gather(ctypes.byref(_sidecar()), 1, None, 16, 16, 16, lay, 1, one, 4, 16, None),
         SR_ERR_NULL_ARG),
        (lib.sr_anchor_gather(ctypes.byref(_sidecar()), 1, 16, 16, 16, 16, lay, 1, one, 4, None, None),
         SR_ERR_NULL_ARG),
        (lib.sr_anchor_gather(ctypes.byref(_sidecar()), 70000, 16, 16, 16, 16, lay, 1, one, 4, 16, None),
         SR_ERR_BAD_SHAPE),
    ]
    for i, (got, want) in enumerate(cases):
        assert got == want, (i, got, want)


# -------------------------------------------------------------------- GPU
def _dev(a):
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    elif a.dtype == np.uint32:
        a = a.view(np.int32)
    return torch.from_numpy(a).cuda()


def _host(t, dtype):
    return t.cpu().numpy().view(dtype)


def _log(msg):
    print(msg, flush=True)


@pytest.mark.gpu
@pytest.mark.parametrize("n,density", [(0, 0.1), (1, 1.0), (8191, 0.07), (8192, 0.0), (8193, 1.0),
                                       (100000, 1 / 16), (70001, 0.5)])
def test_compact_matches_oracle(n, density):
    import torch
    _log(f"compact n={n} density={density}")
    rng = np.random.default_rng(n)
    dest = np.where(rng.random(n) < density, rng.integers(0, 1 << 20, n), -1).astype(np.int32)
    d_dest = _dev(dest) if n else torch.zeros(1, dtype=torch.int32, device="cuda")
    sel = torch.full((max(n, 1),), -7, dtype=torch.int32, device="cuda")
    n_sel = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    sr.LIB.sr_anchor_compact(d_dest.data_ptr(), n, sel.data_ptr(), n_sel.data_ptr(),
                             torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    want = paged.compact(dest)
    k = int(n_sel.item())
    assert k == len(want)
    assert np.array_equal(sel[:k].cpu().numpy(), want)
    assert bool((sel[k:] == -7).all())


def _write_and_compare(c, d, eb, compact):
    import torch
    dest = paged.dest_table(c.positions, c.token_req, c.page_tables(), wsc.PAGE, wsc.PER_PAGE)
    want = paged.anchor_write(c.pool, c.hidden, dest, wsc.PER_PAGE)
    pool = _dev(c.pool)
    hidden = [_dev(h) for h in c.hidden]
    d_dest = _dev(dest)
    sc = sr.make_sidecar(pool, c.n_layers, wsc.PER_PAGE, d)
    if compact:
        sel = torch.empty(len(dest), dtype=torch.int32, device="cuda")
        n_sel = torch.empty(1, dtype=torch.int32, device="cuda")
        sr.anchor_compact(d_dest, sel, n_sel)
        sr.anchor_write(sc, hidden, d_dest, sel, n_sel)
    else:
        sr.anchor_write(sc, hidden, d_dest)
    torch.cuda.synchronize()
    got = _host(pool, want.dtype)
    assert np.array_equal(got, want)


@pytest.mark.gpu
@pytest.mark.parametrize("compact", [True, False])
@pytest.mark.parametrize("seed,spans,n_layers,d,eb,holes", [
    (0, [(0, 1000), (0, 64), (0, 59), (0, 4096)], 7, 2560, 2, 0.0),    # prefill, Qwen3.5-4B rows
    (1, [(128, 700), (63, 64), (60, 61), (5000, 5001)], 3, 64, 4, 0.3),  # chunks + decode, fp32 rows, holes
    (2, [(0, 300)] * 5, 2, 8, 2, 0.0),                                  # 16-byte rows
])
def test_write_matches_oracle(compact, seed, spans, n_layers, d, eb, holes):
    _log(f"write seed={seed} compact={compact} layers={n_layers} d={d} eb={eb}")
    c = wsc.write_case(seed, spans, n_layers, d, eb, holes)
    _write_and_compare(c, d, eb, compact)


def _gather_and_compare(g, d, layers, t_cap=None):
    import torch
    want, want_cu = paged.anchor_gather(g.pool, g.n_layers, wsc.PER_PAGE, g.block_tables(), g.anchor_first,
                                        g.n_anchors, layers)
    T = int(want_cu[-1])
    cap = T if t_cap is None else t_cap
    pool = _dev(g.pool)
    sc = sr.make_sidecar(pool, g.n_layers, wsc.PER_PAGE, d)
    fill = np.uint16(0xBEEF) if g.pool.dtype == np.uint16 else np.uint32(0xDEADBEEF)
    outs = [_dev(np.full((max(cap, 1), d), fill, dtype=g.pool.dtype)) for _ in layers]
    cu = torch.full((len(g.n_anchors) + 1,), -7, dtype=torch.int32, device="cuda")
    if cap == 0:
        outs = [o[:0] for o in outs]
    bt = g.block_table if g.block_table.size else np.zeros(1, np.int32)   # a table with no pages
    sr.anchor_gather(sc, _dev(bt), _dev(g.block_cu), _dev(g.anchor_first), _dev(g.n_anchors), layers, outs, cu)
    torch.cuda.synchronize()
    assert np.array_equal(cu.cpu().numpy(), want_cu)
    for o, w in zip(outs, want):
        got = _host(o, g.pool.dtype)
        n = min(cap, T)
        assert np.array_equal(got[:n], w[:n])
        assert (got[n:cap] == fill).all()


@pytest.mark.gpu
@pytest.mark.parametrize("seed,ks,n_layers,d,eb,layers", [
    (0, [17, 0, 4, 1, 33, 0], 7, 2560, 2, [6, 0, 3]),      # ragged, empty requests, layers out of order
    (1, [1], 1, 8, 2, [0]),
    (2, [64, 128, 3], 2, 64, 4, [1, 0]),                   # fp32 rows
    (3, [0, 0, 0], 2, 64, 2, [1]),                         # nothing to replay
    (4, [5] * 300, 3, 64, 2, [2]),                         # many requests (a wave's rows span several)
])
def test_gather_matches_oracle(seed, ks, n_layers, d, eb, layers):
    _log(f"gather seed={seed} reqs={len(ks)} layers={layers} d={d} eb={eb}")
    g = wsc.gather_case(seed, ks, n_layers, d, eb)
    _gather_and_compare(g, d, layers)


@pytest.mark.gpu
def test_gather_stops_at_the_output_capacity():
    _log("gather with t_cap short of the total")
    g = wsc.gather_case(5, [40, 7, 30], 2, 64, 2)
    _gather_and_compare(g, 64, [1, 0], t_cap=50)


@pytest.mark.gpu
def test_gather_full_varlen16_group():
    """The 16-request workload's replay suffixes (36,672 anchors), all 7
    anchored layers of Qwen3.5-4B rows: the launch configuration bench.py
    times for the gather."""
    import workloads as W
    wl = W.make_config("varlen16")
    _log("gather varlen16 x 7 layers")
    g = wsc.gather_case(0, wl.seg_lens, 7, 2560, 2)
    _gather_and_compare(g, 2560, list(range(7)))


@pytest.mark.gpu
def test_write_then_gather_returns_the_hidden_rows():
    """Round trip: a prefill written through the device write path, then its
    last k anchors gathered on the device, are the hidden rows at those
    requests' last k sampled positions."""
    import torch
    _log("write then gather round trip")
    spans = [(0, 640), (0, 1000), (0, 64)]
    c = wsc.write_case(9, spans, 2, 64, 2)
    dest = paged.dest_table(c.positions, c.token_req, c.page_tables(), wsc.PAGE, wsc.PER_PAGE)
    pool = _dev(c.pool)
    sc = sr.make_sidecar(pool, 2, wsc.PER_PAGE, 64)
    d_dest = _dev(dest)
    sel = torch.empty(len(dest), dtype=torch.int32, device="cuda")
    n_sel = torch.empty(1, dtype=torch.int32, device="cuda")
    sr.anchor_compact(d_dest, sel, n_sel)
    sr.anchor_write(sc, [_dev(h) for h in c.hidden], d_dest, sel, n_sel)
    n_total = [4 * (b // 64) + max(0, b % 64 - 60) for _, b in spans]
    ks = [min(n, 9) for n in n_total]
    first = [n - k for n, k in zip(n_total, ks)]
    tables = c.page_tables()
    bt = np.concatenate([np.array(t, np.int32) for t in tables])
    bcu = np.concatenate([[0], np.cumsum([len(t) for t in tables])]).astype(np.int32)
    outs = [_dev(np.zeros((sum(ks), 64), np.uint16)) for _ in range(2)]
    cu = torch.empty(len(spans) + 1, dtype=torch.int32, device="cuda")
    sr.anchor_gather(sc, _dev(bt), _dev(bcu), _dev(np.array(first, np.int32)), _dev(np.array(ks, np.int32)),
                     [0, 1], outs, cu)
    torch.cuda.synchronize()
    cu_h = cu.cpu().numpy()
    for r in range(len(spans)):
        idx = [i for i in range(len(c.positions)) if c.token_req[i] == r and c.positions[i] % 64 >= 60]
        want = idx[len(idx) - ks[r]:]
        for l in range(2):
            got = _host(outs[l], np.uint16)[cu_h[r]:cu_h[r + 1]]
            assert np.array_equal(got, c.hidden[l][want])


@pytest.mark.gpu
def test_write_and_gather_replay_under_hip_graph_capture():
    """Section 5.1 moves the anchor writes into the captured graph of each
    serving step.  The compaction, the indexed copy and the gather are
    stream-ordered and allocate nothing, so one graph holds all three; every
    replay (with eager work and synchronisation between replays, and the
    outputs poisoned before each) reproduces the oracle bit for bit."""
    import torch
    _log("sidecar calls under graph capture")
    c = wsc.write_case(13, [(0, 700), (128, 900), (60, 61)], 3, 64, 2, hole_frac=0.1)
    dest = paged.dest_table(c.positions, c.token_req, c.page_tables(), wsc.PAGE, wsc.PER_PAGE)
    want_pool = paged.anchor_write(c.pool, c.hidden, dest, wsc.PER_PAGE)
    g = wsc.gather_case(14, [9, 0, 31], 3, 64, 2)
    want_out, want_cu = paged.anchor_gather(g.pool, 3, wsc.PER_PAGE, g.block_tables(), g.anchor_first,
                                            g.n_anchors, [2, 0])
    pool0 = _dev(c.pool)
    pool = pool0.clone()
    hidden = [_dev(h) for h in c.hidden]
    d_dest = _dev(dest)
    sel = torch.empty(len(dest), dtype=torch.int32, device="cuda")
    n_sel = torch.empty(1, dtype=torch.int32, device="cuda")
    sc_w = sr.make_sidecar(pool, 3, wsc.PER_PAGE, 64)
    gpool = _dev(g.pool)
    sc_g = sr.make_sidecar(gpool, 3, wsc.PER_PAGE, 64)
    tabs = [_dev(x) for x in (g.block_table, g.block_cu, g.anchor_first, g.n_anchors)]
    T = int(want_cu[-1])
    outs = [torch.empty((T, 64), dtype=torch.int16, device="cuda") for _ in range(2)]
    cu = torch.empty(4, dtype=torch.int32, device="cuda")
    s = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph, stream=s):
        sr.anchor_compact(d_dest, sel, n_sel, s)
        sr.anchor_write(sc_w, hidden, d_dest, sel, n_sel, s)
        sr.anchor_gather(sc_g, *tabs, [2, 0], outs, cu, s)
    for rep in range(3):
        pool.copy_(pool0)
        for o in outs:
            o.fill_(-1)
        cu.fill_(-7)
        sel.fill_(-7)
        n_sel.fill_(-7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(_host(pool, np.uint16), want_pool), rep
        assert np.array_equal(cu.cpu().numpy(), want_cu), rep
        for o, w in zip(outs, want_out):
            assert np.array_equal(_host(o, np.uint16), w), rep
