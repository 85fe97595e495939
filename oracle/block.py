"""fp64 oracle for group replay chaining (TEST INFRASTRUCTURE ONLY, like all of
``oracle``; it shares no code with the HIP path).

Section 4.1 stores one anchor per group of consecutive linear-attention
layers, the hidden state entering the group, and rebuilds every layer of the
group from it: each replayed layer's output becomes the next layer's input,
and the group never crosses a full-attention layer.  Appendix A counts one
anchor per group (A = G - 1).  Replaying layer j therefore needs, besides its
state, its per-token output and the rest of its transformer block.

The paper prints none of the block's algebra.  Readings (the same ones the
HIP path implements):
  * a block is pre-norm: x = RMSNorm(h) feeds the mixer, h1 = h + mixer(x),
    u = RMSNorm(h1), h_next = h1 + MLP(u); RMSNorm(x) = x / sqrt(mean(x^2) +
    eps) * weight over d_model, eps = 1e-6;
  * the mixer is the Gated DeltaNet layer of oracle/__init__.py with its query
    path: q = W_q x through the same causal conv (q taps conv_q) and SiLU,
    L2-normalised per key head like k and scaled by d_k^-1/2; value head h
    reads query and key head floor(h H_k / H_v);
  * the per-token output reads the state after that token's update:
    o_t = S_t q_t (d_v per value head);
  * an output gate z = W_z x and a per-head RMSNorm over d_v with a weight
    shared by all heads: y = RMSNorm(o) * weight * SiLU(z); mixer(x) = W_o y;
  * the MLP is SwiGLU: W_down (SiLU(W_gate u) * (W_up u)).
"""
from __future__ import annotations

from typing import List, Optional, Tuple

import numpy as np

from . import (causal_depthwise_conv, gated_delta_recurrence, key_head_of, l2_normalize, layer_features, project,
               silu)

__all__ = ["rms_norm", "gated_delta_outputs", "outputs_recurrence", "gdn_mixer", "gated_rms_norm", "swiglu_mlp",
           "block_forward", "replay_group_segment"]


def rms_norm(x: np.ndarray, weight: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * weight over the last axis."""
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * np.asarray(weight, dtype=np.float64)


def gated_delta_outputs(k, v, q, alpha, beta, S0=None) -> Tuple[np.ndarray, np.ndarray]:
    """Gated DeltaNet token by token (Section 2.1, Eq. recurrence) with the
    per-token read-out o_t = S_t q_t.  k, q [L, H, d_k]; v [L, H, d_v];
    alpha, beta [L, H]; S0 [H, d_v, d_k] or None.  Returns (S_L, O [L, H, d_v])."""
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    q = np.asarray(q, dtype=np.float64)
    L, H, dk = k.shape
    dv = v.shape[2]
    S = np.zeros((H, dv, dk)) if S0 is None else np.array(S0, dtype=np.float64)
    O = np.zeros((L, H, dv))
    for t in range(L):
        S = gated_delta_recurrence(k[t:t + 1], v[t:t + 1], alpha[t:t + 1], beta[t:t + 1], S)
        O[t] = np.einsum("hvk,hk->hv", S, q[t])
    return S, O


def outputs_recurrence(k, v, q, alpha, beta, S0=None, impl: str = "auto"):
    """gated_delta_outputs in numpy ("numpy"), or on the plain-C twin ("c";
    "auto": the twin when built).  The two are pinned to each other."""
    from . import crec
    if impl == "c" or (impl == "auto" and crec.available()):
        return crec.recurrence_with_outputs(k, v, q, alpha, beta, S0)
    if impl not in ("numpy", "auto"):
        raise ValueError(impl)
    return gated_delta_outputs(k, v, q, alpha, beta, S0)


def gdn_mixer(shape, blk, x: np.ndarray, impl: str = "auto"):
    """The Gated DeltaNet mixer on normalised inputs x [L, D].  Returns
    (state [H_v, d_k, d_v] = S_L^T, conv tail [C_tail, w-1] with channels
    q | k | v, outputs O [L, H_v, d_v], gate z [L, H_v * d_v])."""
    H_k, H_v, dk, dv, w = shape.n_k_heads, shape.n_v_heads, shape.d_k, shape.d_v, shape.conv_width
    lay = blk.mixer
    x = np.asarray(x, dtype=np.float64)
    L = x.shape[0]
    f = layer_features(shape, lay, x)
    p_q = project(x, lay.w_q)
    qa = silu(causal_depthwise_conv(p_q, blk.conv_q))
    q = l2_normalize(qa.reshape(L, H_k, dk), shape.l2_eps) / np.sqrt(dk)
    kv_head = [key_head_of(h, H_k, H_v) for h in range(H_v)]
    S, O = outputs_recurrence(f["k"][:, kv_head, :], f["v"], q[:, kv_head, :], f["alpha"], f["beta"], impl=impl)
    state = np.transpose(S, (0, 2, 1))
    tail = np.zeros((2 * H_k * dk + H_v * dv, w - 1))
    n_tail = min(L, w - 1)
    if n_tail > 0:
        rows = slice(L - n_tail, L)
        tail[:, w - 1 - n_tail:] = np.concatenate([p_q[rows], f["p_k"][rows], f["p_v"][rows]], axis=1).T
    z = project(x, blk.w_z)
    return state, tail, O, z


def gated_rms_norm(o: np.ndarray, z: np.ndarray, weight: np.ndarray, eps: float) -> np.ndarray:
    """Per value head: RMSNorm of o over d_v (shared weight) times SiLU(z).
    o [L, H_v, d_v], z [L, H_v * d_v]; returns [L, H_v * d_v]."""
    L, H, dv = o.shape
    y = rms_norm(o, weight, eps) * silu(np.asarray(z, dtype=np.float64).reshape(L, H, dv))
    return y.reshape(L, H * dv)


def swiglu_mlp(u: np.ndarray, w_gate, w_up, w_down) -> np.ndarray:
    """W_down (SiLU(W_gate u) * (W_up u)) for rows u [L, D]."""
    return project(silu(project(u, w_gate)) * project(u, w_up), w_down)


def block_forward(shape, blk, h: np.ndarray, eps: float = 1e-6, impl: str = "auto"):
    """One pre-norm block on its input rows h [L, D].  Returns (h_next,
    state, tail, y) with y the gated, normalised mixer output [L, H_v d_v]."""
    h = np.asarray(h, dtype=np.float64)
    x = rms_norm(h, blk.ln_in, eps)
    state, tail, O, z = gdn_mixer(shape, blk, x, impl=impl)
    y = gated_rms_norm(O, z, blk.norm_o, eps)
    h1 = h + project(y, blk.w_o)
    h_next = h1 + swiglu_mlp(rms_norm(h1, blk.ln_post, eps), blk.w_gate, blk.w_up, blk.w_down)
    return h_next, state, tail, y


def replay_group_segment(shape, blocks, x: np.ndarray, eps: float = 1e-6,
                         impl: str = "auto") -> Tuple[List[Tuple[np.ndarray, np.ndarray]], List[np.ndarray]]:
    """Rebuilds every layer of a group from one segment's group-entry anchors
    x [L, D] (Section 4.1).  Returns ([(state, tail)] per layer, [input rows
    of each layer]).  The last layer's block output is not needed (a
    full-attention layer follows) and is not formed."""
    h = np.asarray(x, dtype=np.float64)
    out, inputs = [], []
    for j, blk in enumerate(blocks):
        inputs.append(h)
        if j + 1 < len(blocks):
            h, state, tail, _ = block_forward(shape, blk, h, eps, impl=impl)
        else:
            state, tail, _, _ = gdn_mixer(shape, blk, rms_norm(h, blk.ln_in, eps), impl=impl)
        out.append((state, tail))
    return out, inputs
