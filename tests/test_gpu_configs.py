"""GPU parity on the five named workloads at their full sizes, in the launch
configuration the benchmark times (one call over all segments and layers).
The oracle recomputes sampled (layer, segment) slabs one by one; the small
workloads are checked in full."""
import numpy as np
import pytest
import torch

import workloads as W
from gpu_harness import check_pairs, log, run, upload

pytestmark = pytest.mark.gpu


def _sampled(wl, k_extra=1, seed=0):
    lens = np.array(wl.seg_lens)
    pick = {int(np.argmin(lens)), int(np.argmax(lens))}
    r = np.random.default_rng(seed)
    while len(pick) < min(len(lens), 2 + k_extra):
        pick.add(int(r.integers(len(lens))))
    return sorted(pick)


def _run_config(name):
    log(f"{name}: generating inputs")
    wl = W.make_config(name)
    log(f"{name}: T={wl.t_total}, layers={len(wl.layers)}, segments={len(wl.seg_lens)}; uploading")
    dev = upload(wl)
    log(f"{name}: replay on GPU")
    run(dev)
    for ns in dev.layers:
        assert not torch.any(torch.isnan(ns.state_out)), "a live slot was not written"
    return wl, dev


def test_tiny_fp32_full():
    wl, dev = _run_config("tiny")
    check_pairs(dev, [(0, 0)])


def test_gdn_single_full():
    wl, dev = _run_config("gdn_single")
    check_pairs(dev, [(0, 0)])


def test_varlen16_sampled():
    wl, dev = _run_config("varlen16")
    check_pairs(dev, [(0, b) for b in _sampled(wl, 1)])


def test_multilayer12_fp8_sampled():
    wl, dev = _run_config("multilayer12")
    check_pairs(dev, [(0, 0), (11, 3), (5, 1)])


def test_stress64_long_memory_sampled():
    wl, dev = _run_config("stress64")
    check_pairs(dev, [(0, b) for b in _sampled(wl, 0)])
