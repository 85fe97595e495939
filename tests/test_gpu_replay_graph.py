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
    cases = [([70, 5, 129], None, 0), ([300, 400, 7], [2, -1, 0], 1), ([1000, 1500, 600, 3], None, 2),
             ([70, 5, 129], None, 0), ([20] * 10, None, -1), ([0, 33], None, 0)]
    for seg, slots, bucket in cases:
        log(f"graph replay: segments {seg}, slots {slots}, expected bucket {bucket}")
        wl, dev = _batch(shape, seg, slots)
        run(dev)                                   # eager reference into dev's own outputs
        ref_s, ref_t = dev.layers[0].state_out, dev.layers[0].tail_out
        for rep in range(2):
            state.fill_(float("nan"))
            tail.fill_(float("nan"))
            g.anchors(0)[:wl.t_total].copy_(dev.layers[0].anchors.view(torch.int16))
            torch.cuda.synchronize()
            used = g.run(len(seg), wl.t_total, dev.cu_seqlens, dev.slot_ids if slots else None)
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
