"""Graph-bucketed replay (sr_replay_graph.h): batches padded to their bucket
with sentinel segments and replayed from captured graphs must write exactly
what an eager sr_replay_state call writes for the same batch (no row's
arithmetic depends on the padding), on every replay of a bucket's graph, and
batches with more segments than the graph holds must take the eager path."""
import numpy as np
import pytest
import torch

import workloads as W
from gpu_harness import log, run, upload

pytestmark = pytest.mark.gpu

SLOTS = 16


def _batch(shape, seg, slot_ids=None):
    wl = W.make_workload("rgraph", shape, seg, seed=5, slot_ids=slot_ids or list(range(len(seg))), n_slots=SLOTS)
    dev = upload(wl)
    return wl, dev


def test_graph_buckets_match_eager_replay():
    import paper_2609_33477_amd as sr
    shape = W.Shape(256, 2, 4, 128, 128)
    base_wl, base = _batch(shape, [64])
    layers = [sr.LayerTensors(**vars(ns)) for ns in base.layers]
    g = sr.ReplayGraph(shape, layers, max_segments=8, bucket_rows=[256, 1024, 4096])
    state, tail = base.layers[0].state_out, base.layers[0].tail_out
    # (segments, slots, expected bucket); -1: eager (too many segments, or more
    # rows than the largest bucket: then on the caller's anchors and workspace)
    cases = [([70, 5, 129], None, 0), ([300, 400, 7], [2, -1, 0], 1), ([1000, 1500, 600, 3], None, 2),
             ([70, 5, 129], None, 0), ([20] * 10, None, -1), ([0, 33], None, 0), ([3000, 2000, 5], None, -1)]
    for seg, slots, bucket in cases:
        log(f"graph replay: segments {seg}, slots {slots}, expected bucket {bucket}")
        wl, dev = _batch(shape, seg, slots)
        ws = run(dev)                              # eager reference into dev's own outputs
        ref_s, ref_t = dev.layers[0].state_out, dev.layers[0].tail_out
        over = wl.t_total > g.max_rows
        for rep in range(2):
            state.fill_(float("nan"))
            tail.fill_(float("nan"))
            if not over:
                g.anchors(0)[:wl.t_total].copy_(dev.layers[0].anchors.view(torch.int16))
            torch.cuda.synchronize()
            used = g.run(len(seg), wl.t_total, dev.cu_seqlens, dev.slot_ids if slots else None,
                         eager_anchors=[dev.layers[0].anchors] if over else None,
                         eager_workspace=ws if over else None)
            torch.cuda.synchronize()
            assert used == bucket, (seg, used)
            for b, slot in enumerate(wl.slot_ids):
                if slot < 0:
                    continue
                assert torch.equal(state[slot], ref_s[slot]), (seg, rep, b)
                assert torch.equal(tail[slot], ref_t[slot]), (seg, rep, b)
            live = {s for s in wl.slot_ids if s >= 0}
            for s in range(SLOTS):
                if s not in live:
                    assert torch.all(torch.isnan(state[s])), (seg, s)
    # an over-long batch without caller anchors is refused before any launch
    import paper_2609_33477_amd.binding as B
    with pytest.raises(B.SrError) as e:
        g.run(1, 5000, torch.tensor([0, 5000], dtype=torch.int32, device="cuda"))
    assert e.value.status == 2
    g.close()


def test_pipelined_fetch_and_replay_of_two_groups():
    """Two groups (objects) of two layers each, sharing one lent workspace and
    replayed in order on one stream, with each group's anchors fetched from
    pinned host memory on a copy stream (group 1's fetch overlaps group 0's
    replay).  Two batches in a row: the second batch's fetch into a group must
    wait for that group's first replay.  A consumer stream waits on the
    groups' hand-off events.  Every state and tail equals the eager replay of
    the same batch."""
    import paper_2609_33477_amd as sr
    shape = W.Shape(256, 2, 4, 128, 128)
    n_groups, per_group = 2, 2
    rows_max = 1024
    bases = [W.make_workload(f"grp{gi}", shape, [64], n_layers=per_group, seed=40 + gi, n_slots=SLOTS)
             for gi in range(n_groups)]
    devs = [upload(b) for b in bases]
    ws = torch.empty(sr.replay_workspace_size(shape, per_group, rows_max), dtype=torch.uint8, device="cuda")
    graphs = [sr.ReplayGraph(shape, [sr.LayerTensors(**vars(ns)) for ns in d.layers], max_segments=6,
                             bucket_rows=[256, rows_max], workspace=ws) for d in devs]
    replay_stream, copy_stream, consumer = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    batches = [([100, 7, 300], [3, 0, 9]), ([500, 1, 64, 200], [1, 2, -1, 4])]
    for bi, (seg, slots) in enumerate(batches):
        wls = [W.make_workload(f"grp{gi}", shape, seg, n_layers=per_group, seed=40 + gi, slot_ids=slots,
                               n_slots=SLOTS) for gi in range(n_groups)]
        refs = [upload(w) for w in wls]
        for r in refs:
            run(r)                                            # eager references
        host = [[r.layers[li].anchors.view(torch.int16).cpu().pin_memory() for li in range(per_group)]
                for r in refs]
        cu, sl = refs[0].cu_seqlens, refs[0].slot_ids
        for d in devs:
            for ns in d.layers:
                ns.state_out.fill_(float("nan"))
                ns.tail_out.fill_(float("nan"))
        torch.cuda.synchronize()
        t_total = sum(seg)
        for gi, g in enumerate(graphs):
            g.fetch([(host[gi][li], li, 0) for li in range(per_group)], copy_stream)
            used = g.run(len(seg), t_total, cu, sl, stream=replay_stream)
            assert used == (0 if t_total <= 256 else 1)
            g.wait(consumer)
        done = torch.cuda.Event()
        done.record(consumer)
        done.synchronize()
        torch.cuda.synchronize()
        log(f"pipelined batch {bi}: segments {seg}")
        for gi in range(n_groups):
            for li in range(per_group):
                for b, slot in enumerate(slots):
                    if slot < 0:
                        continue
                    assert torch.equal(devs[gi].layers[li].state_out[slot], refs[gi].layers[li].state_out[slot])
                    assert torch.equal(devs[gi].layers[li].tail_out[slot], refs[gi].layers[li].tail_out[slot])
    for g in graphs:
        g.close()


def test_graph_replay_matches_oracle():
    """Graph-replayed states and tails against the fp64 oracle directly (not
    only against the eager path), for two batches in two buckets."""
    import paper_2609_33477_amd as sr
    from gpu_harness import TOL_BF16, check_slab
    from workloads.device import to_device
    shape = W.Shape(256, 2, 4, 128, 128)
    base_wl, base = _batch(shape, [64])
    layers = [sr.LayerTensors(**vars(ns)) for ns in base.layers]
    g = sr.ReplayGraph(shape, layers, max_segments=8, bucket_rows=[256, 1024])
    state, tail = base.layers[0].state_out, base.layers[0].tail_out
    for seg, slots in (([70, 5, 129, 0], [4, 1, 9, 2]), ([300, 1, 400, 64], [0, -1, 3, 7])):
        # seed 5 as in _batch: the same layer weights as the graph's layers
        wl = W.make_workload("rgraph_oracle", shape, seg, seed=5, slot_ids=slots, n_slots=SLOTS)
        state.fill_(float("nan"))
        tail.fill_(float("nan"))
        g.anchors(0)[:wl.t_total].copy_(to_device(wl.layers[0].anchors, "bf16").view(torch.int16))
        cu = torch.from_numpy(wl.cu_seqlens).cuda()
        sl = torch.tensor(slots, dtype=torch.int32, device="cuda")
        torch.cuda.synchronize()
        used = g.run(len(seg), wl.t_total, cu, sl)
        torch.cuda.synchronize()
        log(f"graph vs oracle: segments {seg}, bucket {used}")
        for b, slot in enumerate(slots):
            if slot < 0:
                continue
            check_slab(wl, 0, b, state[slot].cpu().numpy(), tail[slot].float().cpu().numpy(), TOL_BF16)
    g.close()


def test_graph_keeps_layer_tensors_alive():
    """The captured graphs freeze the layers' pointers, so the object must hold
    the tensors even after the caller drops its references."""
    import gc
    import weakref
    import paper_2609_33477_amd as sr
    shape = W.Shape(128, 1, 1, 32, 32)
    _, dev = _batch(shape, [8])
    layers = [sr.LayerTensors(**vars(ns)) for ns in dev.layers]
    refs = [weakref.ref(layers[0].w_k), weakref.ref(layers[0].state_out)]
    g = sr.ReplayGraph(shape, layers, max_segments=2, bucket_rows=[64])
    del layers, dev
    gc.collect()
    assert all(r() is not None for r in refs)
    g.close()
