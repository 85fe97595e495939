"""GPU parity of heads whose key and value widths differ (Appendix A:
OLMo-Hybrid-7B, d_k = 96, d_v = 192) against the fp64 oracle: the fused
projection with key heads and value halves padded to 128 columns and the
pipelined bf16 scan running each value head as two units (an even number
of value heads), and the unfused bf16 path (projection GEMM,
one-head-per-wave conv/gates, the q-tail blocks on their own, the
state-only chunk kernel; an odd number).  Ragged and empty segments, sentinel slots, fp8
weights, a short conv, fp32 conv taps and tail, an initial state, bitwise
determinism, and the model's full shape."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_harness import TOL_BF16, check_pairs, log, rel_frob, run, upload

pytestmark = pytest.mark.gpu

RAGGED = [1, 3, 64, 65, 200, 0, 130, 127]


def _live_pairs(wl):
    return [(li, b) for li in range(len(wl.layers)) for b in range(len(wl.seg_lens))
            if wl.slot_ids[b] >= 0 and wl.seg_lens[b] > 0]


def test_rect_heads_ragged_two_layers():
    shape = W.Shape(256, 2, 2, 96, 192)
    wl = W.make_workload("rect", shape, RAGGED, n_layers=2, seed=301)
    log(f"rect heads 96x192 ragged: T={wl.t_total}, 2 layers")
    dev = upload(wl)
    run(dev)
    check_pairs(dev, _live_pairs(wl), TOL_BF16)
    b0 = RAGGED.index(0)
    for li in range(2):
        assert torch.all(dev.layers[li].state_out[b0] == 0)
        assert torch.all(dev.layers[li].tail_out[b0] == 0)


def test_rect_heads_odd_value_heads_unfused():
    # 3 value heads of 192 columns do not fill whole 128-column blocks: the
    # unfused path, with GQA (one key head)
    shape = W.Shape(256, 1, 3, 96, 192)
    seg = [40, 0, 131, 7]
    wl = W.make_workload("rect_odd", shape, seg, seed=309)
    log(f"rect heads, 3 value heads (unfused): T={wl.t_total}")
    dev = upload(wl)
    run(dev)
    check_pairs(dev, _live_pairs(wl), TOL_BF16)
    assert torch.all(dev.layers[0].state_out[1] == 0)


def test_rect_heads_fp8_gqa_sentinels_short_conv():
    shape = W.Shape(384, 2, 4, 96, 192, weight_dtype=W.FP8, conv_width=3)
    seg = [70, 2, 129, 40]
    wl = W.make_workload("rect_fp8", shape, seg, seed=303, slot_ids=[4, -1, 0, 2], n_slots=6)
    log(f"rect heads fp8 weights, GQA, sentinel, w=3: T={wl.t_total}")
    dev = upload(wl)
    run(dev)
    check_pairs(dev, _live_pairs(wl), TOL_BF16)
    live = {s for s in wl.slot_ids if s >= 0}
    for s in range(wl.n_slots):
        if s not in live:
            assert torch.all(torch.isnan(dev.layers[0].state_out[s])), s


def test_rect_heads_fp32_conv_and_tail_without_q():
    shape = W.Shape(256, 2, 2, 96, 192, conv_dtype=W.F32, tail_dtype=W.F32)
    wl = W.make_workload("rect_f32conv", shape, [5, 131, 66], seed=305)
    log(f"rect heads, fp32 conv taps and tail, no q tail: T={wl.t_total}")
    dev = upload(wl, with_q=False)
    run(dev)
    check_pairs(dev, _live_pairs(wl), TOL_BF16)


def test_rect_heads_initial_state_and_determinism():
    shape = W.Shape(256, 2, 2, 96, 192)
    seg = [3, 150]
    wl = W.make_workload("rect_init", shape, seg, seed=307)
    S0 = np.random.default_rng(3).standard_normal((2, 2, 96, 192)).astype(np.float32) * 0.5
    dev = upload(wl, state_in=[S0])
    ws = run(dev)
    first = dev.layers[0].state_out.clone()
    run(dev, workspace=ws)
    assert torch.equal(first, dev.layers[0].state_out)
    cu = wl.cu_seqlens
    L = wl.layers[0]
    for b in range(2):
        ref, _ = oracle.replay_segment(shape, L, L.anchors[cu[b]:cu[b + 1]], S0=S0[b].astype(np.float64))
        err = rel_frob(first[b].cpu().numpy(), ref)
        log(f"rect heads with initial state, seg {b}: {err:.3e}")
        assert err <= TOL_BF16


def test_olmo_hybrid_shape():
    """OLMo-Hybrid-7B's linear-layer shape: d_model 3840, 30 key and 30 value
    heads, d_k = 96, d_v = 192."""
    shape = W.Shape(3840, 30, 30, 96, 192)
    wl = W.make_workload("olmo", shape, [300, 129, 64, 1], seed=309)
    log(f"OLMo-Hybrid shape: T={wl.t_total}")
    dev = upload(wl)
    run(dev)
    check_pairs(dev, _live_pairs(wl), TOL_BF16)


def test_rect_heads_graph_and_noalloc_match_eager():
    """The graph-bucketed replay and the allocation-free entry point take the
    rectangular-head path through the same sr_replay_state: each must write
    what the eager call writes, bit for bit (graph: twice, into NaN)."""
    import paper_2609_33477_amd as sr
    shape = W.Shape(256, 2, 2, 96, 192)
    seg = [70, 0, 129]
    wl = W.make_workload("rect_graph", shape, seg, seed=311, n_slots=4)
    log(f"rect heads through a graph and the no-alloc entry: T={wl.t_total}")
    dev = upload(wl)
    run(dev)
    L0 = dev.layers[0]
    ref_s, ref_t = L0.state_out.clone(), L0.tail_out.clone()
    live = [s for s in wl.slot_ids if s >= 0]
    layers = [sr.LayerTensors(**vars(ns)) for ns in dev.layers]
    g = sr.ReplayGraph(shape, layers, max_segments=4, bucket_rows=[256, 512])
    g.anchors(0)[:wl.t_total].copy_(L0.anchors.view(torch.int16))
    for rep in range(2):
        L0.state_out.fill_(float("nan"))
        L0.tail_out.fill_(float("nan"))
        torch.cuda.synchronize()
        used = g.run(len(seg), wl.t_total, dev.cu_seqlens, dev.slot_ids)
        torch.cuda.synchronize()
        assert used == 0
        for s in live:
            assert torch.equal(L0.state_out[s], ref_s[s]), (rep, s)
            assert torch.equal(L0.tail_out[s], ref_t[s]), (rep, s)
    g.close()
    L0.state_out.fill_(float("nan"))
    L0.tail_out.fill_(float("nan"))
    sr.replay_state_noalloc(shape, layers, len(seg), wl.t_total, dev.cu_seqlens, dev.slot_ids)
    torch.cuda.synchronize()
    for s in live:
        assert torch.equal(L0.state_out[s], ref_s[s]), s
        assert torch.equal(L0.tail_out[s], ref_t[s]), s
