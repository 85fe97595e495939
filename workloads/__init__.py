"""Seeded synthetic inputs for SuffixReplay state reconstruction.

This module is shared by the fp64 oracle and by the tests/bench that drive the
HIP library, and it holds none of the method's arithmetic: it only draws random
numbers, rounds them to the storage formats the layer keeps (bf16, OCP fp8
E4M3 with a per-output-channel bf16 scale, fp32), and describes the workload
shapes.

Every array is returned as float32 whose values are exactly representable in
the declared storage dtype, so the oracle (which upcasts to fp64) and the GPU
path (which converts to bf16 / float8_e4m3fn) see bit-identical inputs.

Shapes follow the Gated DeltaNet linear-attention layers of the paper's models
(Appendix A, Table "Model parameters and the resulting sizes"): the 16-request
varlen workload has Qwen3.5-4B's linear-layer shape (d=2560, H_k/H_v = 16/32,
d_k = d_v = 128) and the multi-layer workload Qwen3.6-27B's (d=5120, 16/48).
Replay lengths are whole 64-token pages (Section 4.2 aligns anchors to
64-token pages).
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Dict, List, Optional

import numpy as np

F32 = "f32"
BF16 = "bf16"
FP8 = "fp8_e4m3"

# Largest finite OCP E4M3 magnitude (S.1111.110 = 1.75 * 2^8).
E4M3_MAX = 448.0


# --------------------------------------------------------------------------
# storage-format rounding
# --------------------------------------------------------------------------
def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); float32 out."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) & np.uint32(0xFFFF0000)).view(np.float32)


def round_to_e4m3(x: np.ndarray) -> np.ndarray:
    """Round to the nearest OCP FP8 E4M3 value (ties to even), saturating at
    +-448; float32 out.  E4M3: bias 7, 3 mantissa bits, subnormal step 2^-9."""
    xd = np.asarray(x, dtype=np.float64)
    ax = np.minimum(np.abs(xd), E4M3_MAX)
    _, e = np.frexp(ax)                       # ax = m * 2^e, m in [0.5, 1)
    step = np.ldexp(1.0, e - 4)               # 3 mantissa bits below the lead
    step = np.maximum(step, 2.0 ** -9)        # subnormal spacing
    q = np.minimum(np.rint(ax / step) * step, E4M3_MAX)
    return (np.sign(xd) * q).astype(np.float32)


def quantize_rows_e4m3(w: np.ndarray):
    """Per-output-channel (row) fp8 quantisation: s = bf16(max|w_row| / 448),
    q = e4m3(w / s).  Returns (q values, s values), both float32, with
    q * s the dequantised weight."""
    amax = np.max(np.abs(w), axis=1).astype(np.float32)
    s = round_to_bf16(np.maximum(amax / np.float32(E4M3_MAX), np.float32(2.0 ** -30)))
    q = round_to_e4m3(w / s[:, None])
    return q, s


def _store(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == F32:
        return np.ascontiguousarray(x, dtype=np.float32)
    if dtype in (BF16, FP8):  # fp8 matrices are produced by quantize_rows_e4m3
        return round_to_bf16(x)
    raise ValueError(dtype)


# --------------------------------------------------------------------------
# workload description
# --------------------------------------------------------------------------
@dataclass
class Shape:
    d_model: int
    n_k_heads: int
    n_v_heads: int
    d_k: int
    d_v: int
    conv_width: int = 4
    l2_eps: float = 1e-6
    anchor_dtype: str = BF16
    weight_dtype: str = BF16   # projection weights (q, k, v, a, b)
    conv_dtype: str = BF16     # depthwise conv taps
    tail_dtype: str = BF16     # conv-tail output
    recurrence: str = "gdn"    # "gdn" (decay + erase) or "decay" (per-head decay only)

    @property
    def c_kv(self) -> int:     # conv channels the recurrence consumes (k | v)
        return self.n_k_heads * self.d_k + self.n_v_heads * self.d_v

    @property
    def c_tail(self) -> int:   # conv-state channels q | k | v (Appendix A)
        return 2 * self.n_k_heads * self.d_k + self.n_v_heads * self.d_v

    @property
    def n_proj(self) -> int:   # projection width k | v | a | b
        return self.c_kv + 2 * self.n_v_heads


@dataclass
class LayerInputs:
    anchors: np.ndarray                 # [T, D]
    w_q: np.ndarray                     # [H_k*d_k, D]
    w_k: np.ndarray                     # [H_k*d_k, D]
    w_v: np.ndarray                     # [H_v*d_v, D]
    w_a: np.ndarray                     # [H_v, D]  decay-gate input
    w_b: np.ndarray                     # [H_v, D]  erase-strength input
    conv_w: np.ndarray                  # [C_kv, w] (k channels, then v)
    a_log: np.ndarray                   # [H_v]
    dt_bias: np.ndarray                 # [H_v]
    # fp8 only: per-output-channel bf16 scales, keyed "q","k","v","a","b"
    w_scale: Optional[Dict[str, np.ndarray]] = None


@dataclass
class Workload:
    name: str
    description: str
    shape: Shape
    seg_lens: List[int]
    slot_ids: List[int]
    n_slots: int
    layers: List[LayerInputs] = field(default_factory=list)
    seed: int = 0

    @property
    def t_total(self) -> int:
        return int(sum(self.seg_lens))

    @property
    def cu_seqlens(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.seg_lens)]).astype(np.int32)

    @property
    def max_seqlen(self) -> int:
        return int(max(self.seg_lens)) if self.seg_lens else 0

    @property
    def replayed_tokens(self) -> int:
        """Anchor rows replayed by one call, summed over layers and live
        segments (sentinel segments are excluded)."""
        live = sum(L for L, s in zip(self.seg_lens, self.slot_ids) if s >= 0)
        return live * len(self.layers)


# Each tensor is drawn from its own stream, seeded by (workload seed, layer,
# tensor id), so a tensor -- or a prefix of its rows -- can be drawn without
# drawing the others.
TENSOR_IDS = {"anchors": 0, "q": 1, "k": 2, "v": 3, "a": 4, "b": 5, "conv": 6,
              "a_log": 7, "dt_bias": 8}
SEGMENT_STREAM = 1000


def tensor_rng(seed: int, layer: int, name: str) -> np.random.Generator:
    return np.random.default_rng((seed, layer, TENSOR_IDS[name]))


def draw_anchors(seed: int, layer: int, rows: int, shape: Shape) -> np.ndarray:
    """Anchors h ~ N(0, 1) rounded to the anchor dtype; drawing fewer rows
    yields a prefix of the full draw."""
    g = tensor_rng(seed, layer, "anchors")
    return _store(g.standard_normal((rows, shape.d_model), dtype=np.float32), shape.anchor_dtype)


def _draw_layer(seed: int, layer: int, shape: Shape, t_total: int,
                dt_bias_mean: float, dt_bias_std: float = 0.5,
                weight_std: float = 0.02) -> LayerInputs:
    D = shape.d_model
    qk = shape.n_k_heads * shape.d_k
    vv = shape.n_v_heads * shape.d_v
    hv = shape.n_v_heads

    def normal(name, rows, cols, std):
        g = tensor_rng(seed, layer, name)
        return g.standard_normal((rows, cols), dtype=np.float32) * np.float32(std)

    anchors = draw_anchors(seed, layer, t_total, shape)
    raw = {
        "q": normal("q", qk, D, weight_std),
        "k": normal("k", qk, D, weight_std),
        "v": normal("v", vv, D, weight_std),
        "a": normal("a", hv, D, weight_std),
        "b": normal("b", hv, D, weight_std),
    }
    conv_w = _store(normal("conv", shape.c_kv, shape.conv_width, weight_std), shape.conv_dtype)
    a_log = tensor_rng(seed, layer, "a_log").uniform(np.log(1.0), np.log(16.0), size=hv).astype(np.float32)
    z = tensor_rng(seed, layer, "dt_bias").standard_normal(hv, dtype=np.float32)
    dt_bias = (np.float32(dt_bias_mean) + np.float32(dt_bias_std) * z).astype(np.float32)

    if shape.weight_dtype == FP8:
        mats, scales = {}, {}
        for key, w in raw.items():
            mats[key], scales[key] = quantize_rows_e4m3(w)
    else:
        mats = {key: _store(w, shape.weight_dtype) for key, w in raw.items()}
        scales = None
    return LayerInputs(anchors=anchors, w_q=mats["q"], w_k=mats["k"], w_v=mats["v"],
                       w_a=mats["a"], w_b=mats["b"], conv_w=conv_w, a_log=a_log,
                       dt_bias=dt_bias, w_scale=scales)


def make_workload(name: str, shape: Shape, seg_lens, n_layers: int = 1, seed: int = 0,
                  slot_ids=None, n_slots: Optional[int] = None,
                  dt_bias_mean: float = 0.0, description: str = "") -> Workload:
    """Explicit workload: fixed segment lengths, seeded layer draws."""
    seg_lens = [int(x) for x in seg_lens]
    if slot_ids is None:
        slot_ids = list(range(len(seg_lens)))
    slot_ids = [int(s) for s in slot_ids]
    if n_slots is None:
        n_slots = max([s + 1 for s in slot_ids if s >= 0], default=0)
    t_total = int(sum(seg_lens))
    layers = [_draw_layer(seed, li, shape, t_total, dt_bias_mean) for li in range(n_layers)]
    return Workload(name=name, description=description, shape=shape, seg_lens=seg_lens,
                    slot_ids=slot_ids, n_slots=n_slots, layers=layers, seed=seed)


def _page_lengths(rng: np.random.Generator, n: int, lo: int, hi: int, page: int = 64):
    """Uniform over whole pages: page * U{lo/page .. hi/page}."""
    return [int(page * x) for x in rng.integers(lo // page, hi // page, size=n, endpoint=True)]


# dt_bias mean for the long-memory workload, chosen so the empirical mean decay
# alpha over all (row, head) of the generated inputs is 0.995.  It is derived by
# tests/golden/derive_long_memory_dt_bias.py (which evaluates the gates with the
# oracle) and checked by a CPU test.
LONG_MEMORY_DT_BIAS_MEAN = -7.494

CONFIG_NAMES = ("tiny", "gdn_single", "varlen16", "multilayer12", "stress64")


# Variants of a named workload: same seed and tensors, another recurrence.
VARIANTS = {"varlen16_decay": ("varlen16", "decay")}

# Workloads beyond the five: OLMo-Hybrid-7B's linear-layer shape (Appendix A:
# d_model 3840, 30 key and 30 value heads, d_k = 96, d_v = 192) on
# varlen16's length distribution.
EXTRA_SEEDS = {"olmo_varlen": 6}


def _config_table(name: str):
    if name in VARIANTS:
        base, rec = VARIANTS[name]
        seed, shape, seg, n_layers, mu = _config_table(base)
        return seed, replace(shape, recurrence=rec), seg, n_layers, mu
    seed = EXTRA_SEEDS[name] if name in EXTRA_SEEDS else CONFIG_NAMES.index(name) + 1
    rng = np.random.default_rng((seed, SEGMENT_STREAM))
    if name == "tiny":
        shape = Shape(128, 2, 2, 32, 32, anchor_dtype=F32, weight_dtype=F32,
                      conv_dtype=F32, tail_dtype=F32)
        return seed, shape, [256], 1, 0.0
    if name == "gdn_single":
        return seed, Shape(2048, 16, 16, 128, 128), [2048], 1, 0.0
    if name == "varlen16":
        return seed, Shape(2560, 16, 32, 128, 128), _page_lengths(rng, 16, 512, 4096), 1, 0.0
    if name == "multilayer12":
        return seed, Shape(5120, 16, 48, 128, 128, weight_dtype=FP8), [4096] * 4, 12, 0.0
    if name == "stress64":
        return (seed, Shape(4096, 32, 32, 128, 128), _page_lengths(rng, 64, 1024, 8192), 1,
                LONG_MEMORY_DT_BIAS_MEAN)
    if name == "olmo_varlen":
        return seed, Shape(3840, 30, 30, 96, 192), _page_lengths(rng, 16, 512, 4096), 1, 0.0
    raise KeyError(name)


def config_shape(name: str):
    """(shape, segment lengths, layer count) of a named workload, without
    drawing its tensors."""
    _, shape, seg, n_layers, _ = _config_table(name)
    return shape, seg, n_layers


def make_config(name: str) -> Workload:
    """The five named workloads (seed = position in CONFIG_NAMES + 1).

    tiny          1 request, 1 layer, D=128, H=2, d=32, L=256, fp32
    gdn_single    1 request, D=2048, H=16, d=128, L=2048, bf16
    varlen16      16 requests, L ~ 64*U{8..64}, D=2560, H_k=16, H_v=32, bf16
    multilayer12  12 layers x 4 requests x L=4096, D=5120, H_k=16, H_v=48,
                  fp8 E4M3 weights + per-channel bf16 scales, bf16 anchors
    stress64      64 requests, L ~ 64*U{16..128}, D=4096, H=32, bf16,
                  dt_bias shifted so mean alpha is 0.995
    varlen16_decay  varlen16's inputs under the per-head-decay recurrence
    olmo_varlen   16 requests, L ~ 64*U{8..64}, D=3840, H=30, d_k=96, d_v=192,
                  bf16 (OLMo-Hybrid-7B's linear layers)
    Weights ~ N(0, 0.02), anchors ~ N(0, 1), A_log ~ U(log 1, log 16),
    dt_bias ~ N(mu, 0.5), zero initial state.
    """
    seed, shape, seg, n_layers, mu = _config_table(name)
    layers = [_draw_layer(seed, li, shape, int(sum(seg)), mu) for li in range(n_layers)]
    return Workload(name=name, description=name, shape=shape, seg_lens=seg,
                    slot_ids=list(range(len(seg))), n_slots=len(seg), layers=layers, seed=seed)
