"""GPU parity on the five named workloads at their full sizes, in the launch
configuration the benchmark times (one call over all segments and layers).

Every live (layer, segment) slab is compared with the fp64 oracle: the
relative Frobenius error of the whole [H_v][d_k][d_v] state, of each value
head, and of the conv tail.  The GPU runs once per workload (a module-level
cache holds its outputs on the host); the oracle work of the large workloads
is split over several tests so that each finishes in well under a minute on
the host cores (projection on the BLAS threads, recurrence on the oracle's C
twin, one thread per value head)."""
import numpy as np
import pytest
import torch

import workloads as W
from gpu_harness import check_slab, log, run, tolerance, upload

pytestmark = pytest.mark.gpu

_CACHE = {}


def _gpu_outputs(name):
    """(workload, states [layers][slots][H_v][d_k][d_v], tails) of one GPU
    call over the whole workload, on the host."""
    if name in _CACHE:
        return _CACHE[name]
    _CACHE.clear()                      # one workload's inputs on the host at a time
    log(f"{name}: generating inputs")
    wl = W.make_config(name)
    log(f"{name}: T={wl.t_total}, layers={len(wl.layers)}, segments={len(wl.seg_lens)}; uploading")
    dev = upload(wl)
    log(f"{name}: replay on GPU")
    run(dev)
    states = [ns.state_out.cpu().numpy() for ns in dev.layers]
    tails = [ns.tail_out.float().cpu().numpy() for ns in dev.layers]
    del dev
    torch.cuda.empty_cache()
    for li, st in enumerate(states):
        assert not np.any(np.isnan(st)), f"layer {li}: a live slot was not written"
    _CACHE[name] = (wl, states, tails)
    return _CACHE[name]


def _check(name, pairs):
    wl, states, tails = _gpu_outputs(name)
    tol = tolerance(wl)
    worst = np.zeros(3)
    for li, b in pairs:
        slot = wl.slot_ids[b]
        worst = np.maximum(worst, check_slab(wl, li, b, states[li][slot], tails[li][slot], tol))
    log(f"{name}: {len(pairs)} slabs, worst state {worst[0]:.3e}, worst head {worst[1]:.3e}, "
        f"worst tail {worst[2]:.3e} (tolerance {tol:g}, per head {2 * tol:g})")


def test_tiny_fp32_all_slabs():
    _check("tiny", [(0, 0)])


def test_gdn_single_all_slabs():
    _check("gdn_single", [(0, 0)])


def test_varlen16_all_slabs():
    _check("varlen16", [(0, b) for b in range(16)])


@pytest.mark.parametrize("part", range(4))
def test_multilayer12_fp8_all_slabs(part):
    _check("multilayer12", [(li, b) for li in range(3 * part, 3 * part + 3) for b in range(4)])


@pytest.mark.parametrize("part", range(4))
def test_stress64_long_memory_all_slabs(part):
    _check("stress64", [(0, b) for b in range(part, 64, 4)])
