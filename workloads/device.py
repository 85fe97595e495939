"""Upload a generated workload to the GPU as the tensors the C ABI expects.

Plumbing only: float32 arrays whose values are exact in their storage dtype
are converted to bf16 / float8_e4m3fn / fp32 device tensors, and output and
workspace buffers are allocated.  No arithmetic of the method happens here.
"""
from __future__ import annotations

from dataclasses import dataclass
from types import SimpleNamespace
from typing import List, Optional

import numpy as np
import torch

from . import BF16, F32, FP8, Workload

TORCH_DTYPES = {F32: torch.float32, BF16: torch.bfloat16, FP8: torch.float8_e4m3fn}


def to_device(x: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(device)
    return t.to(TORCH_DTYPES[dtype]).contiguous()


@dataclass
class DeviceWorkload:
    wl: Workload
    layers: List[SimpleNamespace]        # attribute names as sr_layer
    cu_seqlens: torch.Tensor
    slot_ids: Optional[torch.Tensor]
    with_q: bool

    @property
    def n_segments(self) -> int:
        return len(self.wl.seg_lens)


def upload(wl: Workload, with_q: bool = True, state_in: Optional[List[np.ndarray]] = None,
           out_fill: float = float("nan"), device="cuda", explicit_slots: bool = True) -> DeviceWorkload:
    """Device copies of every layer tensor plus state/tail outputs prefilled
    with ``out_fill`` (NaN by default, so unwritten slots stay visible)."""
    sh = wl.shape
    layers = []
    for li, L in enumerate(wl.layers):
        ns = SimpleNamespace()
        ns.anchors = to_device(L.anchors, sh.anchor_dtype, device)
        for name in ("k", "v", "a", "b", "q"):
            ns.__dict__["w_" + name] = to_device(getattr(L, "w_" + name), sh.weight_dtype, device)
            ns.__dict__["s_" + name] = (to_device(L.w_scale[name], BF16, device)
                                         if L.w_scale is not None else None)
        if not with_q:
            ns.w_q = None
            ns.s_q = None
        ns.conv_w = to_device(L.conv_w, sh.conv_dtype, device)
        ns.a_log = to_device(L.a_log, F32, device)
        ns.dt_bias = to_device(L.dt_bias, F32, device)
        ns.state_in = None if state_in is None else to_device(state_in[li], F32, device)
        ns.state_out = torch.full((wl.n_slots, sh.n_v_heads, sh.d_k, sh.d_v), out_fill,
                                  dtype=torch.float32, device=device)
        c_tail = (sh.c_tail if with_q else sh.c_kv)
        ns.tail_out = torch.full((wl.n_slots, c_tail, sh.conv_width - 1), out_fill,
                                 dtype=TORCH_DTYPES[sh.tail_dtype], device=device)
        layers.append(ns)
    cu = torch.from_numpy(wl.cu_seqlens).to(device)
    slots = torch.tensor(wl.slot_ids, dtype=torch.int32, device=device) if explicit_slots else None
    return DeviceWorkload(wl=wl, layers=layers, cu_seqlens=cu, slot_ids=slots, with_q=with_q)


@dataclass
class DeviceGroup:
    gw: object                           # workloads.group.GroupWorkload
    blocks: List[SimpleNamespace]        # attribute names as sr_block
    anchors: torch.Tensor
    cu_seqlens: torch.Tensor
    slot_ids: Optional[torch.Tensor]


def upload_group(gw, out_fill: float = float("nan"), device="cuda") -> DeviceGroup:
    """Device copies of a group workload's anchors and block tensors, with
    state and tail outputs prefilled with ``out_fill``.  The block's conv taps
    are the q taps followed by the mixer's k | v taps ([C_tail][w])."""
    sh = gw.shape
    blocks = []
    for b in gw.blocks:
        m = b.mixer
        ns = SimpleNamespace()
        for name in ("q", "k", "v", "a", "b"):
            setattr(ns, "w_" + name, to_device(getattr(m, "w_" + name), BF16, device))
        ns.w_z = to_device(b.w_z, BF16, device)
        ns.conv_w = to_device(np.concatenate([b.conv_q, m.conv_w]), sh.conv_dtype, device)
        ns.a_log = to_device(m.a_log, F32, device)
        ns.dt_bias = to_device(m.dt_bias, F32, device)
        for name in ("norm_o", "w_o", "ln_in", "ln_post", "w_gate", "w_up", "w_down"):
            setattr(ns, name, to_device(getattr(b, name), BF16, device))
        ns.state_out = torch.full((gw.n_slots, sh.n_v_heads, sh.d_k, sh.d_v), out_fill, dtype=torch.float32,
                                  device=device)
        ns.tail_out = torch.full((gw.n_slots, sh.c_tail, sh.conv_width - 1), out_fill,
                                 dtype=TORCH_DTYPES[sh.tail_dtype], device=device)
        blocks.append(ns)
    cu = torch.from_numpy(gw.cu_seqlens).to(device)
    slots = torch.tensor(gw.slot_ids, dtype=torch.int32, device=device)
    return DeviceGroup(gw=gw, blocks=blocks, anchors=to_device(gw.anchors, BF16, device), cu_seqlens=cu,
                       slot_ids=slots)
