"""GPU parity of the HIP replay path against the fp64 oracle on small seeded
inputs that span several GEMM tiles, several 64-row scan chunks and ragged
tails, plus the behaviour the C ABI promises (sentinel slots, empty
segments, initial state, determinism, varlen invariance, graph capture).
Everything goes through the C ABI via the ctypes binding."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
import paper_2609_33477_amd as sr
from gpu_harness import TOL_BF16, TOL_F32, check_pairs, check_slab, layer_tensors, log, rel_frob, run, upload

pytestmark = pytest.mark.gpu

RAGGED = [1, 3, 64, 65, 200, 0, 130, 127]


def _live_pairs(wl):
    return [(li, b) for li in range(len(wl.layers)) for b in range(len(wl.seg_lens))
            if wl.slot_ids[b] >= 0 and wl.seg_lens[b] > 0]


@pytest.mark.parametrize("d", [32, 64, 128])
def test_bf16_ragged_segments(d):
    shape = W.Shape(256, 2, 4, d, d)
    wl = W.make_workload(f"bf16_d{d}", shape, RAGGED, seed=11 + d)
    log(f"bf16 ragged d={d}: T={wl.t_total}")
    dev = upload(wl)
    run(dev)
    check_pairs(dev, _live_pairs(wl), TOL_BF16)
    # the empty segment yields a zero state and a zero tail
    b0 = RAGGED.index(0)
    assert torch.all(dev.layers[0].state_out[b0] == 0)
    assert torch.all(dev.layers[0].tail_out[b0] == 0)


@pytest.mark.parametrize("d", [32, 128])
def test_fp32_ragged_segments(d):
    shape = W.Shape(128, 2, 2, d, d, anchor_dtype=W.F32, weight_dtype=W.F32, conv_dtype=W.F32,
                    tail_dtype=W.F32)
    wl = W.make_workload(f"f32_d{d}", shape, [5, 64, 100, 1, 190], seed=21 + d)
    log(f"fp32 ragged d={d}: T={wl.t_total}")
    dev = upload(wl)
    run(dev)
    check_pairs(dev, _live_pairs(wl), TOL_F32)


def test_fp8_weights_gqa():
    shape = W.Shape(320, 2, 6, 128, 128, weight_dtype=W.FP8)
    wl = W.make_workload("fp8", shape, [70, 129, 2], n_layers=2, seed=31)
    log(f"fp8 weights: T={wl.t_total}, 2 layers")
    dev = upload(wl)
    run(dev)
    check_pairs(dev, _live_pairs(wl), TOL_BF16)


def test_without_q_tail_and_short_conv():
    shape = W.Shape(192, 1, 2, 64, 64, conv_width=2)
    wl = W.make_workload("noq", shape, [1, 66, 9], seed=41)
    dev = upload(wl, with_q=False)
    run(dev)
    check_pairs(dev, _live_pairs(wl), TOL_BF16)


def test_sentinel_slots_untouched_and_slot_mapping():
    shape = W.Shape(256, 2, 4, 128, 128)
    seg = [40, 65, 7, 130]
    wl = W.make_workload("slots", shape, seg, seed=51, slot_ids=[3, -1, 0, -5], n_slots=5)
    dev = upload(wl)
    run(dev)
    out = dev.layers[0].state_out
    for s in (1, 2, 4):           # never written: still the NaN fill
        assert torch.all(torch.isnan(out[s])), s
        assert torch.all(torch.isnan(dev.layers[0].tail_out[s].float())), s
    check_pairs(dev, [(0, 0), (0, 2)], TOL_BF16)


def test_identity_slots_when_slot_ids_null():
    shape = W.Shape(256, 2, 2, 128, 128)
    wl = W.make_workload("nullslots", shape, [33, 80], seed=52)
    dev = upload(wl, explicit_slots=False)
    assert dev.slot_ids is None
    run(dev)
    check_pairs(dev, [(0, 0), (0, 1)], TOL_BF16)


def test_initial_state_and_contraction_bound():
    """state_in path against the oracle, and the contraction bound of the
    replayed state: ||S(S0) - S(0)||_F <= ||S0||_F * prod(alpha)."""
    shape = W.Shape(256, 2, 2, 128, 128)
    seg = [3, 90]
    wl = W.make_workload("init", shape, seg, seed=61)
    r = np.random.default_rng(0)
    S0 = r.standard_normal((2, 2, 128, 128)).astype(np.float32) * 0.5
    dev0 = upload(wl)
    run(dev0)
    dev1 = upload(wl, state_in=[S0])
    run(dev1)
    cu = wl.cu_seqlens
    L = wl.layers[0]
    for b in range(2):
        x = L.anchors[cu[b]:cu[b + 1]]
        ref, _ = oracle.replay_segment(shape, L, x, S0=S0[b].astype(np.float64))
        got = dev1.layers[0].state_out[b].cpu().numpy()
        assert rel_frob(got, ref) <= TOL_BF16
        f = oracle.layer_features(shape, L, x)
        diff = (dev1.layers[0].state_out[b] - dev0.layers[0].state_out[b]).double().cpu().numpy()
        for h in range(2):
            bound = np.linalg.norm(S0[b, h]) * np.prod(f["alpha"][:, h])
            assert np.linalg.norm(diff[h]) <= bound * (1 + 1e-2) + 1e-6 * np.linalg.norm(S0[b, h])


def test_deterministic_and_varlen_invariant():
    """Bitwise-identical results across calls, and a packed batch equals each
    segment replayed alone (no cross-segment leakage in conv or scan)."""
    shape = W.Shape(256, 2, 4, 128, 128)
    seg = [100, 1, 64, 77]
    wl = W.make_workload("det", shape, seg, seed=71)
    dev = upload(wl)
    run(dev)
    first = dev.layers[0].state_out.clone()
    first_tail = dev.layers[0].tail_out.clone()
    run(dev)
    assert torch.equal(first, dev.layers[0].state_out)
    assert torch.equal(first_tail, dev.layers[0].tail_out)
    cu = wl.cu_seqlens
    for b in range(len(seg)):
        single = W.Workload(name="one", description="", shape=shape, seg_lens=[seg[b]], slot_ids=[0], n_slots=1,
                            layers=[W.LayerInputs(**{**vars(wl.layers[0]),
                                                     "anchors": wl.layers[0].anchors[cu[b]:cu[b + 1]]})])
        d1 = upload(single)
        run(d1)
        assert torch.equal(d1.layers[0].state_out[0], first[b]), b
        assert torch.equal(d1.layers[0].tail_out[0], first_tail[b]), b


def test_hip_graph_capture_replays():
    """The call is stream-ordered and allocation-free, so it can be captured;
    every replay of the graph must reproduce the eager result."""
    shape = W.Shape(256, 2, 4, 128, 128)
    wl = W.make_workload("graph", shape, [70, 5, 129], seed=81)
    dev = upload(wl)
    ws = run(dev)
    eager = dev.layers[0].state_out.clone()
    eager_tail = dev.layers[0].tail_out.clone()
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=s):
        run(dev, workspace=ws, stream=s, sync=False)
    for _ in range(3):
        dev.layers[0].state_out.fill_(float("nan"))
        dev.layers[0].tail_out.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(dev.layers[0].state_out, eager)
        assert torch.equal(dev.layers[0].tail_out, eager_tail)


def test_fp32_conv_weights_and_tail_with_bf16_anchors():
    """The fused projection with fp32 conv weights and an fp32 conv tail (the
    taps and the tail are the dtype-dependent parts of its epilogue)."""
    shape = W.Shape(256, 2, 4, 128, 128, conv_dtype=W.F32, tail_dtype=W.F32)
    wl = W.make_workload("convf32", shape, [70, 5, 131], seed=81)
    log(f"fp32 conv/tail: T={wl.t_total}")
    dev = upload(wl)
    run(dev)
    check_pairs(dev, _live_pairs(wl), TOL_BF16)


def test_no_decay_keeps_the_initial_state():
    """alpha = 1 to fp32 precision (A_log = -40): nothing may decay the
    carried state, across many 32-row steps and with a nonzero state_in."""
    shape = W.Shape(256, 2, 2, 64, 64)
    wl = W.make_workload("nodecay", shape, [300, 45], seed=91)
    wl.layers[0].a_log[:] = -40.0
    r = np.random.default_rng(1)
    S0 = r.standard_normal((2, 2, 64, 64)).astype(np.float32)
    dev = upload(wl, state_in=[S0])
    run(dev)
    cu = wl.cu_seqlens
    L = wl.layers[0]
    for b in range(2):
        ref, _ = oracle.replay_segment(shape, L, L.anchors[cu[b]:cu[b + 1]], S0=S0[b].astype(np.float64))
        got = dev.layers[0].state_out[b].cpu().numpy()
        err = rel_frob(got, ref)
        log(f"no decay seg {b}: state rel err {err:.3e}")
        assert err <= TOL_BF16


def test_more_segments_than_the_device_sort():
    """Over 256 segments the scan takes work units in segment order instead
    of sorting them longest-first; results must not depend on that."""
    shape = W.Shape(128, 1, 2, 32, 32)
    seg = [int(x) for x in np.random.default_rng(5).integers(0, 40, size=300)]
    wl = W.make_workload("manyseg", shape, seg, seed=95)
    log(f"{len(seg)} segments, T={wl.t_total}")
    dev = upload(wl)
    run(dev)
    live = [p for p in _live_pairs(wl)]
    check_pairs(dev, live[::17] + live[-3:], TOL_BF16)


# Every (dtype, head size, conv width) combination the host accepts, on a
# small ragged batch, so that no accepted combination goes untested.
COMBOS = [
    # (name, shape keyword arguments, d, conv width, with q tail)
    ("f32_d64", dict(anchor_dtype=W.F32, weight_dtype=W.F32, conv_dtype=W.F32, tail_dtype=W.F32), 64, 4, True),
    ("f32_bf16_conv_tail", dict(anchor_dtype=W.F32, weight_dtype=W.F32, conv_dtype=W.BF16, tail_dtype=W.BF16),
     64, 4, True),
    ("fp8_d32", dict(weight_dtype=W.FP8), 32, 4, True),
    ("fp8_d64", dict(weight_dtype=W.FP8), 64, 4, True),
    ("bf16_w1", dict(), 64, 1, True),
    ("bf16_w3", dict(), 64, 3, True),
    ("f32_w3", dict(anchor_dtype=W.F32, weight_dtype=W.F32, conv_dtype=W.F32, tail_dtype=W.F32), 32, 3, True),
    ("f32_w1", dict(anchor_dtype=W.F32, weight_dtype=W.F32, conv_dtype=W.F32, tail_dtype=W.F32), 32, 1, False),
    ("fp8_w2_noq", dict(weight_dtype=W.FP8, tail_dtype=W.F32), 128, 2, False),
]


@pytest.mark.parametrize("name,kw,d,w,with_q", COMBOS, ids=[c[0] for c in COMBOS])
def test_accepted_combinations(name, kw, d, w, with_q):
    shape = W.Shape(192, 2, 4, d, d, conv_width=w, **kw)
    wl = W.make_workload(name, shape, [1, 2, 70, 0, 131], seed=200 + [c[0] for c in COMBOS].index(name))
    log(f"combination {name}: T={wl.t_total}")
    dev = upload(wl, with_q=with_q)
    run(dev)
    tol = TOL_F32 if shape.anchor_dtype == W.F32 else TOL_BF16
    check_pairs(dev, _live_pairs(wl), tol, check_tail=w > 1)
    b0 = 3
    assert torch.all(dev.layers[0].state_out[b0] == 0)


def test_mixed_layers_share_projection_launches():
    """The fused projections of up to four layers of a call share a launch;
    five layers (a launch of four, then one) whose tails differ: layer 1
    without W_q (a k | v tail), layer 3 without a tail.  Every state and
    tail matches the oracle, and each layer's state is bit for bit the one a
    call of that layer alone gives."""
    shape = W.Shape(256, 2, 4, 128, 128)
    seg = [70, 1, 200, 33]
    wl = W.make_workload("mixed_layers", shape, seg, n_layers=5, seed=97)
    dev = upload(wl)
    dev.layers[1].w_q = None
    dev.layers[1].tail_out = torch.full((wl.n_slots, shape.c_kv, shape.conv_width - 1), float("nan"),
                                        dtype=torch.bfloat16, device="cuda")
    dev.layers[3].tail_out = None
    log(f"mixed layers: T={wl.t_total}, 5 layers")
    run(dev)
    for li in range(5):
        for b in range(len(seg)):
            slot = wl.slot_ids[b]
            got_state = dev.layers[li].state_out[slot].cpu().numpy()
            tail = dev.layers[li].tail_out
            got_tail = tail[slot].float().cpu().numpy() if tail is not None else None
            check_slab(wl, li, b, got_state, got_tail, TOL_BF16, with_q=(li != 1), check_tail=tail is not None)
    ws_bytes = sr.replay_workspace_size(shape, 1, wl.t_total)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    for li in range(5):
        alone = torch.full_like(dev.layers[li].state_out, float("nan"))
        L = sr.LayerTensors(**{**vars(dev.layers[li]), "state_out": alone, "tail_out": None})
        sr.replay_state(shape, [L], len(seg), wl.t_total, dev.cu_seqlens, dev.slot_ids, ws, ws_bytes)
        torch.cuda.synchronize()
        assert torch.equal(alone, dev.layers[li].state_out), li
