"""Helpers for the GPU tests: run the library on an uploaded workload and
compare against the fp64 oracle slab by slab (relative Frobenius norm per
(layer, segment), the metric the tolerances are stated in)."""
from __future__ import annotations

import sys
import time

import numpy as np
import torch

import oracle
import paper_2609_33477_amd as sr
from workloads.device import upload  # noqa: F401  (re-exported for tests)

TOL_F32 = 1e-4
TOL_BF16 = 5e-3


def log(msg: str):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)
    sys.stdout.flush()


def layer_tensors(dev):
    return [sr.LayerTensors(**vars(ns)) for ns in dev.layers]


def run(dev, workspace=None, stream=None, sync=True):
    wl = dev.wl
    ws_bytes = sr.replay_workspace_size(wl.shape, len(wl.layers), wl.t_total)
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device="cuda")
    sr.replay_state(wl.shape, layer_tensors(dev), len(wl.seg_lens), wl.t_total, dev.cu_seqlens,
                    dev.slot_ids, workspace, ws_bytes, stream)
    if sync:
        torch.cuda.synchronize()
    return workspace


def rel_frob(got: np.ndarray, ref: np.ndarray) -> float:
    den = float(np.linalg.norm(ref))
    num = float(np.linalg.norm(np.asarray(got, dtype=np.float64) - ref))
    return num / den if den > 0 else num


def tolerance(wl) -> float:
    return TOL_F32 if wl.shape.anchor_dtype == "f32" else TOL_BF16


def check_pairs(dev, pairs, tol=None, check_tail=True):
    """Oracle vs GPU for (layer, segment) pairs; returns the worst errors."""
    wl = dev.wl
    tol = tolerance(wl) if tol is None else tol
    cu = wl.cu_seqlens
    worst_s = worst_t = 0.0
    for li, b in pairs:
        slot = wl.slot_ids[b]
        assert slot >= 0
        L = wl.layers[li]
        t0 = time.time()
        ref_state, ref_tail = oracle.replay_segment(wl.shape, L, L.anchors[cu[b]:cu[b + 1]], with_q_tail=dev.with_q)
        got_state = dev.layers[li].state_out[slot].cpu().numpy()
        es = rel_frob(got_state, ref_state)
        worst_s = max(worst_s, es)
        msg = f"layer {li} seg {b} (L={wl.seg_lens[b]}, slot {slot}): state rel err {es:.3e}"
        if check_tail and wl.shape.conv_width > 1:
            got_tail = dev.layers[li].tail_out[slot].float().cpu().numpy()
            et = rel_frob(got_tail, ref_tail)
            worst_t = max(worst_t, et)
            msg += f", tail rel err {et:.3e}"
            assert np.all(np.isfinite(got_tail)), msg
        log(msg + f"  [oracle {time.time() - t0:.1f}s]")
        assert np.all(np.isfinite(got_state)), msg
        assert es <= tol, msg
        if check_tail and wl.shape.conv_width > 1:
            assert et <= tol, msg
    return worst_s, worst_t
