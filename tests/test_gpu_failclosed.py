"""Fail-closed replay on the GPU (Section 5.2: a bad input becomes a cache
miss, never a corrupt write).  Each bad varlen table below is rejected by the
device check that runs first in the call: every state and tail stays as it
was (NaN fill), and the reported mask equals the host twin's.  So is the
table of a gather that ran out of output rows.  Every table
here stays inside the allocated buffers even where the check would not stop
it (slot ids below the allocated slot count, row offsets below the allocated
rows), so a broken check shows up as a written output, never as a fault.
A good table afterwards, on the same workspace, replays correctly."""
import numpy as np
import pytest
import torch

import workloads as W
from gpu_harness import TOL_BF16, check_pairs, layer_tensors, log, upload

pytestmark = pytest.mark.gpu

SHAPE = W.Shape(256, 2, 4, 64, 64)
SEG = [40, 65, 7, 88]               # 200 rows
ALLOC_ROWS = 300                    # every buffer holds this many rows
ALLOC_SLOTS = 6

# (name, cu_seqlens, slot_ids, t_total, declared n_slots, expected mask)
BAD = [
    ("bad_start", [5, 40, 105, 112, 200], [0, 1, 2, 3], 200, 4, 1),
    ("not_monotone", [0, 40, 30, 112, 200], [0, 1, 2, 3], 200, 4, 2),
    ("total_short", [0, 40, 105, 112, 190], [0, 1, 2, 3], 200, 4, 4),
    ("total_past_end", [0, 40, 105, 112, 250], [0, 1, 2, 3], 200, 4, 4),
    ("slot_range", [0, 40, 105, 112, 200], [0, 1, 4, 3], 200, 4, 8),
    ("slot_duplicate", [0, 40, 105, 112, 200], [0, 2, 2, 3], 200, 4, 16),
]


def _setup():
    import paper_2609_33477_amd as sr
    wl = W.make_workload("failclosed", SHAPE, SEG + [ALLOC_ROWS - sum(SEG)], seed=3, n_slots=ALLOC_SLOTS)
    dev = upload(wl)
    ws_bytes = sr.replay_workspace_size(SHAPE, 1, ALLOC_ROWS)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    return sr, wl, dev, ws, ws_bytes


@pytest.mark.parametrize("name,cu,slots,t,n_slots,want", BAD, ids=[c[0] for c in BAD])
def test_bad_table_writes_nothing(name, cu, slots, t, n_slots, want):
    sr, wl, dev, ws, ws_bytes = _setup()
    assert sr.validate_varlen_host(cu, slots, t, n_slots) == want
    d_cu = torch.tensor(cu, dtype=torch.int32, device="cuda")
    d_sl = torch.tensor(slots, dtype=torch.int32, device="cuda")
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    log(f"bad table {name}: cu {cu}, slots {slots}, t_total {t}, n_slots {n_slots}")
    sr.replay_state(SHAPE, layer_tensors(dev), 4, t, d_cu, d_sl, ws, ws_bytes, n_slots=n_slots, varlen_status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == want
    assert int(ws[:4].view(torch.int32).item()) == want          # the workspace's flag word
    assert torch.all(torch.isnan(dev.layers[0].state_out))
    assert torch.all(torch.isnan(dev.layers[0].tail_out.float()))
    # the standalone device check agrees
    st2 = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    sr.validate_varlen(d_cu, d_sl, 4, t, n_slots, st2)
    torch.cuda.synchronize()
    assert int(st2.item()) == want
    # the no-alloc entry point is fail-closed the same way
    st3 = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    sr.replay_state_noalloc(SHAPE, layer_tensors(dev), 4, t, d_cu, d_sl, n_slots=n_slots, varlen_status=st3)
    torch.cuda.synchronize()
    assert int(st3.item()) == want
    assert torch.all(torch.isnan(dev.layers[0].state_out))


def test_good_table_after_a_bad_one():
    sr, wl, dev, ws, ws_bytes = _setup()
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    bad_cu = torch.tensor([0, 40, 30, 112, 200], dtype=torch.int32, device="cuda")
    slots = torch.tensor([0, 1, 2, 3], dtype=torch.int32, device="cuda")
    sr.replay_state(SHAPE, layer_tensors(dev), 4, 200, bad_cu, slots, ws, ws_bytes, n_slots=4, varlen_status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 2
    # the whole allocated batch, five segments, through the same workspace
    sr.replay_state(SHAPE, layer_tensors(dev), 5, ALLOC_ROWS, dev.cu_seqlens, dev.slot_ids, ws, ws_bytes,
                    varlen_status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    check_pairs(dev, [(0, b) for b in range(5)], TOL_BF16)


def test_graph_run_with_a_bad_table_writes_nothing():
    import paper_2609_33477_amd as sr
    _, wl, dev, _, _ = _setup()
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    g = sr.ReplayGraph(SHAPE, layer_tensors(dev), max_segments=8, bucket_rows=[256, 512], varlen_status=status)
    g.anchors(0)[:ALLOC_ROWS].copy_(dev.layers[0].anchors.view(torch.int16))
    for cu, slots, want in (([0, 40, 105, 112, 200], [0, 2, 2, 3], 16),      # duplicate slot
                            ([0, 40, 105, 112, 400], [0, 1, 2, 3], 2)):     # rows past the bucket (256)
        torch.cuda.synchronize()
        used = g.run(4, 200, torch.tensor(cu, dtype=torch.int32, device="cuda"),
                     torch.tensor(slots, dtype=torch.int32, device="cuda"))
        torch.cuda.synchronize()
        assert used == 0
        assert int(status.item()) == want, (cu, slots)
        assert torch.all(torch.isnan(dev.layers[0].state_out))
    g.close()


def _to_dev(a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).cuda()


def test_short_gather_is_refused_by_the_replay():
    """The read path end to end: a gather whose outputs hold fewer rows than
    the requests' anchors stops at their capacity but reports the full
    prefix sums; replaying that many rows with its table is refused on the
    device (the table's total is not the row count), so a short gather ends
    as a miss, not as states built from missing rows.  The workspace is
    sized for every row the table names, so nothing could be read outside it
    even without the check."""
    import paper_2609_33477_amd as sr
    from workloads import sidecar as wsc
    _, wl, dev, ws, ws_bytes = _setup()
    cap = 150
    g = wsc.gather_case(11, SEG, 1, SHAPE.d_model, 2)          # 200 anchors of SHAPE's rows
    sc = sr.make_sidecar(_to_dev(g.pool), g.n_layers, wsc.PER_PAGE, SHAPE.d_model)
    rows = torch.zeros((cap, SHAPE.d_model), dtype=torch.int16, device="cuda")
    cu = torch.full((len(SEG) + 1,), -7, dtype=torch.int32, device="cuda")
    log(f"short gather: {sum(SEG)} anchors into {cap} rows, then replay of {cap} rows")
    sr.anchor_gather(sc, _to_dev(g.block_table), _to_dev(g.block_cu), _to_dev(g.anchor_first),
                     _to_dev(g.n_anchors), [0], [rows], cu)
    torch.cuda.synchronize()
    assert cu.cpu().tolist() == [0, 40, 105, 112, 200]
    layers = layer_tensors(dev)
    layers[0] = sr.LayerTensors(**{**vars(dev.layers[0]), "anchors": rows.view(torch.bfloat16)})
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    sr.replay_state(SHAPE, layers, len(SEG), cap, cu, dev.slot_ids[:len(SEG)].contiguous(), ws, ws_bytes,
                    n_slots=ALLOC_SLOTS, varlen_status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == sr.validate_varlen_host(cu.cpu().tolist(), list(range(len(SEG))), cap, ALLOC_SLOTS)
    assert int(status.item()) == 4                               # the total does not match
    assert torch.all(torch.isnan(dev.layers[0].state_out))
    assert torch.all(torch.isnan(dev.layers[0].tail_out.float()))
