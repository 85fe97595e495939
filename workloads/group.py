"""Seeded synthetic inputs for group replay chaining (no arithmetic of the
method: draws, storage rounding and shapes only).

Section 4.1 replays a group of consecutive linear-attention layers from one
stored anchor, the hidden state entering the group; each replayed layer's
block output is the next layer's input.  A block here is a pre-norm
transformer layer around a Gated DeltaNet mixer: the mixer weights of
``workloads.LayerInputs`` plus the q conv taps, the output gate, the output
norm and projection, the two block norms and a SwiGLU MLP of width d_ff.
Every weight is bf16 (values exact in bf16, held as float32), drawn from its
own seeded stream like the single-layer workloads.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List

import numpy as np

from . import BF16, LayerInputs, Shape, _draw_layer, _store

# stream ids of the block tensors, after the mixer's (workloads.TENSOR_IDS)
BLOCK_TENSOR_IDS = {"conv_q": 9, "z": 10, "norm_o": 11, "o": 12, "ln_in": 13, "ln_post": 14, "gate": 15,
                    "up": 16, "down": 17}

# Group shapes (Appendix A's Qwen3.5-4B linear layers: D = 2560, H_k / H_v =
# 16 / 32, d = 128; 24 linear layers in 8 groups, so 3 per group).  The paper
# gives no MLP width; 9728 is the dense MLP width of the Qwen3 4B family.
QWEN35_4B_D_FF = 9728
QWEN35_4B_GROUP_LAYERS = 3


@dataclass
class BlockInputs:
    mixer: LayerInputs          # w_q, w_k, w_v, w_a, w_b, conv_w (k | v), a_log, dt_bias
    conv_q: np.ndarray          # [H_k*d_k, w] conv taps of the q channels
    w_z: np.ndarray             # [H_v*d_v, D] output gate
    norm_o: np.ndarray          # [d_v] weight of the per-head output norm
    w_o: np.ndarray             # [D, H_v*d_v] output projection
    ln_in: np.ndarray           # [D] input norm weight
    ln_post: np.ndarray         # [D] post-mixer norm weight
    w_gate: np.ndarray          # [d_ff, D]
    w_up: np.ndarray            # [d_ff, D]
    w_down: np.ndarray          # [D, d_ff]


@dataclass
class GroupWorkload:
    name: str
    shape: Shape
    d_ff: int
    seg_lens: List[int]
    slot_ids: List[int]
    n_slots: int
    anchors: np.ndarray         # [T, D] group-entry hidden states (bf16 values)
    blocks: List[BlockInputs] = field(default_factory=list)
    norm_eps: float = 1e-6
    seed: int = 0

    @property
    def t_total(self) -> int:
        return int(sum(self.seg_lens))

    @property
    def cu_seqlens(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.seg_lens)]).astype(np.int32)

    @property
    def replayed_tokens(self) -> int:
        live = sum(L for L, s in zip(self.seg_lens, self.slot_ids) if s >= 0)
        return live * len(self.blocks)


def _rng(seed: int, layer: int, name: str) -> np.random.Generator:
    return np.random.default_rng((seed, layer, BLOCK_TENSOR_IDS[name]))


def _draw_block(seed: int, layer: int, shape: Shape, d_ff: int, t_total: int, weight_std: float = 0.02):
    mixer = _draw_layer(seed, layer, shape, t_total if layer == 0 else 0, 0.0, weight_std=weight_std)
    D, qk, vv = shape.d_model, shape.n_k_heads * shape.d_k, shape.n_v_heads * shape.d_v

    def normal(name, rows, cols, std):
        return _store(_rng(seed, layer, name).standard_normal((rows, cols), dtype=np.float32) * np.float32(std), BF16)

    def norm_weight(name, n):
        return _store(1.0 + 0.1 * _rng(seed, layer, name).standard_normal(n, dtype=np.float32), BF16)

    return BlockInputs(mixer=mixer, conv_q=_store(normal("conv_q", qk, shape.conv_width, weight_std), shape.conv_dtype),
                       w_z=normal("z", vv, D, weight_std), norm_o=norm_weight("norm_o", shape.d_v),
                       w_o=normal("o", D, vv, weight_std), ln_in=norm_weight("ln_in", D),
                       ln_post=norm_weight("ln_post", D), w_gate=normal("gate", d_ff, D, weight_std),
                       w_up=normal("up", d_ff, D, weight_std), w_down=normal("down", D, d_ff, weight_std))


def make_group(name: str, shape: Shape, seg_lens, n_layers: int = QWEN35_4B_GROUP_LAYERS,
               d_ff: int = QWEN35_4B_D_FF, seed: int = 0, slot_ids=None, n_slots=None) -> GroupWorkload:
    """A group of n_layers blocks and a packed batch of group-entry anchors
    (N(0, 1) rows rounded to bf16, the first layer's anchor stream)."""
    if shape.anchor_dtype != BF16 or shape.weight_dtype != BF16:
        raise ValueError("group replay workloads are bf16")
    seg_lens = [int(x) for x in seg_lens]
    slot_ids = list(range(len(seg_lens))) if slot_ids is None else [int(s) for s in slot_ids]
    if n_slots is None:
        n_slots = max([s + 1 for s in slot_ids if s >= 0], default=0)
    T = int(sum(seg_lens))
    blocks = [_draw_block(seed, li, shape, d_ff, T) for li in range(n_layers)]
    anchors = blocks[0].mixer.anchors
    return GroupWorkload(name=name, shape=shape, d_ff=d_ff, seg_lens=seg_lens, slot_ids=slot_ids, n_slots=n_slots,
                         anchors=anchors, blocks=blocks, seed=seed)
