"""fp64 CPU oracle for SuffixReplay state reconstruction.

TEST INFRASTRUCTURE ONLY.  Nothing in the library imports this package; only
the test suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may use it.  It shares no code with the HIP path: the only module
both sides use is the seeded input generator ``workloads``.

What it computes (plain, slow, float64, in the paper's order):

* Section 1, Eq. (1)/(2): the recurrent state after position j is a
  deterministic function of the layer inputs h_1..h_j; suffix replay evaluates
  the same function on the last k inputs only, starting from S = 0.  The
  oracle therefore *is* that function, evaluated token by token.
* Section 2.1, Eq. (recurrence): S_t = A_t(S_{t-1}) + B_t, S_0 = 0; A_t and
  B_t are built from linear maps of the layer input h_t (a key, a value and
  two gate inputs).  Gated DeltaNet pairs a decay with a rank-one erase:
  S_t = alpha_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T.
* Appendix A: per value head the state is one d_k x d_v fp32 matrix; the short
  causal convolution over the q, k, v projections (width w) keeps the last
  w-1 *inputs* of its 2 H_k d_k + H_v d_v channels as the conv state.

Readings taken where the paper gives no formula (the paper names the gates but
prints none of their algebra):
  * alpha_t = exp(-exp(A_log) * softplus(a_t + dt_bias)), beta_t = sigmoid(b_t),
    with a_t = W_a h_t, b_t = W_b h_t, one of each per value head;
  * k and v pass through the causal depthwise conv (tap w-1 multiplies the
    current row, no bias, zero history before the replayed suffix), then SiLU;
    k is then L2-normalised per key head: k / sqrt(sum k^2 + eps);
  * value head h reads key head floor(h * H_k / H_v);
  * the state is emitted as M = S^T with layout [H_v][d_k][d_v];
  * the conv tail holds the raw (pre-conv) projections of the last w-1 rows,
    channels ordered q | k | v, layout [C_tail][w-1] oldest -> newest, zero
    where the segment is shorter than w-1.

``shape.recurrence`` selects the state update: "gdn" (the default, above) or
"decay", the per-head decay without the erase that the paper names for
Mamba2 (Section 2.1), kept with Gated DeltaNet's inputs and write.

Parity pins for every function live in tests/test_oracle_pins.py.  The
anchor sidecar's write and read paths (Sections 4.2, 5.1, 5.2) are in
``oracle.paged``, pinned in tests/test_paged_oracle.py.
"""
from __future__ import annotations

from typing import Dict, Optional, Tuple

import numpy as np

__all__ = [
    "project", "causal_depthwise_conv", "silu", "sigmoid", "softplus",
    "l2_normalize", "decay_erase_gates", "key_head_of", "gated_delta_recurrence", "decay_recurrence",
    "replay_segment", "layer_features", "recurrence",
]


def project(x: np.ndarray, w: np.ndarray, scale: Optional[np.ndarray] = None) -> np.ndarray:
    """p = x W^T in fp64 (Section 2.1: the update's key, value and gate inputs
    are linear maps of the layer input).  ``scale`` is a per-output-channel
    multiplier for quantised weights, i.e. W = diag(scale) Q."""
    w64 = np.asarray(w, dtype=np.float64)
    if scale is not None:
        w64 = w64 * np.asarray(scale, dtype=np.float64)[:, None]
    return np.asarray(x, dtype=np.float64) @ w64.T


def causal_depthwise_conv(p: np.ndarray, taps: np.ndarray) -> np.ndarray:
    """Short causal depthwise convolution of width w (Appendix A):
    y[t, c] = sum_{i=0}^{w-1} taps[c, i] * p[t - (w-1) + i, c], with p = 0
    before the first replayed row (replay has no earlier inputs)."""
    p = np.asarray(p, dtype=np.float64)
    taps = np.asarray(taps, dtype=np.float64)
    L = p.shape[0]
    w = taps.shape[1]
    y = np.zeros_like(p)
    for i in range(w):
        lag = w - 1 - i
        if lag < L:
            y[lag:, :] += taps[None, :, i] * p[: L - lag, :]
    return y


def sigmoid(x: np.ndarray) -> np.ndarray:
    """1 / (1 + e^-x) without overflow: with e = e^-|x|, 1 / (1 + e) for
    x >= 0 and e / (1 + e) otherwise."""
    x = np.asarray(x, dtype=np.float64)
    e = np.exp(-np.abs(x))
    r = 1.0 / (1.0 + e)
    return np.where(x >= 0, r, e * r)


def silu(y: np.ndarray) -> np.ndarray:
    y = np.asarray(y, dtype=np.float64)
    return y * sigmoid(y)


def softplus(x: np.ndarray) -> np.ndarray:
    """log(1 + e^x) in the overflow-free form max(x, 0) + log1p(e^-|x|)."""
    x = np.asarray(x, dtype=np.float64)
    return np.maximum(x, 0.0) + np.log1p(np.exp(-np.abs(x)))


def l2_normalize(k: np.ndarray, eps: float) -> np.ndarray:
    """k / sqrt(sum_d k^2 + eps) over the last axis (one key head)."""
    k = np.asarray(k, dtype=np.float64)
    return k / np.sqrt(np.sum(k * k, axis=-1, keepdims=True) + eps)


def decay_erase_gates(a: np.ndarray, b: np.ndarray, a_log: np.ndarray,
                      dt_bias: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Per value head: decay alpha = exp(-exp(A_log) * softplus(a + dt_bias))
    and erase strength beta = sigmoid(b).  ``a``/``b`` are [L, H_v]."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    rate = np.exp(np.asarray(a_log, dtype=np.float64))[None, :]
    alpha = np.exp(-rate * softplus(a + np.asarray(dt_bias, dtype=np.float64)[None, :]))
    beta = sigmoid(b)
    return alpha, beta


def key_head_of(h: int, n_k_heads: int, n_v_heads: int) -> int:
    """Value head h reads key head floor(h * H_k / H_v) (contiguous groups)."""
    return (h * n_k_heads) // n_v_heads


def gated_delta_recurrence(k: np.ndarray, v: np.ndarray, alpha: np.ndarray,
                           beta: np.ndarray, S0: Optional[np.ndarray] = None) -> np.ndarray:
    """Token-by-token Gated DeltaNet recurrence (Section 2.1, Eq. recurrence):

        S_t = alpha_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T

    Arguments are already expanded per value head: k [L, H, d_k],
    v [L, H, d_v], alpha/beta [L, H].  S0 is [H, d_v, d_k] (None = 0).
    Returns S_L as [H, d_v, d_k]."""
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    L, H, dk = k.shape
    dv = v.shape[2]
    S = np.zeros((H, dv, dk)) if S0 is None else np.array(S0, dtype=np.float64)
    for t in range(L):
        kt = k[t]                                   # [H, dk]
        vt = v[t]                                   # [H, dv]
        at = np.asarray(alpha[t], dtype=np.float64)[:, None, None]
        bt = np.asarray(beta[t], dtype=np.float64)[:, None, None]
        Sk = np.einsum("hvk,hk->hv", S, kt)         # S_{t-1} k_t
        S = at * (S - bt * Sk[:, :, None] * kt[:, None, :]) \
            + bt * vt[:, :, None] * kt[:, None, :]
    return S


def decay_recurrence(k: np.ndarray, v: np.ndarray, alpha: np.ndarray,
                     beta: np.ndarray, S0: Optional[np.ndarray] = None) -> np.ndarray:
    """Token-by-token per-head-decay recurrence, the Mamba2-style form the
    paper names beside Gated DeltaNet (Section 2.1, Eq. recurrence: A_t is a
    per-head decay, no erase), with the same write as Gated DeltaNet:

        S_t = alpha_t S_{t-1} + beta_t v_t k_t^T

    Arguments and result as gated_delta_recurrence."""
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    L, H, dk = k.shape
    dv = v.shape[2]
    S = np.zeros((H, dv, dk)) if S0 is None else np.array(S0, dtype=np.float64)
    for t in range(L):
        at = np.asarray(alpha[t], dtype=np.float64)[:, None, None]
        bt = np.asarray(beta[t], dtype=np.float64)[:, None, None]
        S = at * S + bt * v[t][:, :, None] * k[t][:, None, :]
    return S


RECURRENCES = {"gdn": gated_delta_recurrence, "decay": decay_recurrence}


def recurrence(kind: str, k, v, alpha, beta, S0=None, impl: str = "auto") -> np.ndarray:
    """The recurrence ``kind`` ("gdn" or "decay") over expanded per-head inputs
    (arguments as gated_delta_recurrence).  ``impl`` "numpy" runs the numpy
    loops above, "c" the plain-C twin in oracle/recurrence.c (one host thread
    per head), "auto" the C twin when it is built.  The two are pinned to each
    other; the C twin only makes full-size workloads affordable."""
    from . import crec
    if impl == "c" or (impl == "auto" and crec.available()):
        return crec.recurrence(kind, k, v, alpha, beta, S0)
    if impl not in ("numpy", "auto"):
        raise ValueError(impl)
    return RECURRENCES[kind](k, v, alpha, beta, S0)


def layer_features(shape, layer, x: np.ndarray) -> Dict[str, np.ndarray]:
    """Projection, conv, SiLU, key norm and gates for one segment's rows x
    ([L, D]).  Returns k [L, H_k, d_k], v [L, H_v, d_v], alpha/beta [L, H_v]
    and the raw k|v projections."""
    H_k, H_v, dk, dv = shape.n_k_heads, shape.n_v_heads, shape.d_k, shape.d_v
    sc = layer.w_scale or {}
    L = x.shape[0]
    p_k = project(x, layer.w_k, sc.get("k"))
    p_v = project(x, layer.w_v, sc.get("v"))
    a = project(x, layer.w_a, sc.get("a"))
    b = project(x, layer.w_b, sc.get("b"))
    act = silu(causal_depthwise_conv(np.concatenate([p_k, p_v], axis=1), layer.conv_w))
    k = l2_normalize(act[:, : H_k * dk].reshape(L, H_k, dk), shape.l2_eps)
    v = act[:, H_k * dk:].reshape(L, H_v, dv)
    alpha, beta = decay_erase_gates(a, b, layer.a_log, layer.dt_bias)
    return {"k": k, "v": v, "alpha": alpha, "beta": beta, "p_k": p_k, "p_v": p_v}


def replay_segment(shape, layer, x: np.ndarray, S0: Optional[np.ndarray] = None,
                   with_q_tail: bool = True, impl: str = "auto") -> Tuple[np.ndarray, np.ndarray]:
    """Replay one segment's anchors x [L, D] through one linear layer.

    Returns (state [H_v, d_k, d_v] = S_L^T, tail [C_tail, w-1]).  ``S0`` is an
    optional initial state in the same [H_v, d_k, d_v] layout (None = zero, the
    method).  With ``with_q_tail`` False the tail holds only k | v channels.
    ``impl`` selects the recurrence implementation (see ``recurrence``)."""
    H_k, H_v, dk, dv = shape.n_k_heads, shape.n_v_heads, shape.d_k, shape.d_v
    w = shape.conv_width
    x = np.asarray(x, dtype=np.float64)
    L = x.shape[0]
    c_tail = (2 * H_k * dk if with_q_tail else H_k * dk) + H_v * dv
    tail = np.zeros((c_tail, w - 1))
    if L == 0:
        state = np.zeros((H_v, dk, dv)) if S0 is None else np.array(S0, dtype=np.float64)
        return state, tail

    f = layer_features(shape, layer, x)
    kv_head = [key_head_of(h, H_k, H_v) for h in range(H_v)]
    k_per_v = f["k"][:, kv_head, :]                                  # [L, H_v, dk]
    S0_s = None if S0 is None else np.transpose(np.asarray(S0, dtype=np.float64), (0, 2, 1))
    S = recurrence(getattr(shape, "recurrence", "gdn"), k_per_v, f["v"], f["alpha"], f["beta"], S0_s, impl=impl)
    state = np.transpose(S, (0, 2, 1))                               # M = S^T

    n_tail = min(L, w - 1)
    rows = slice(L - n_tail, L)
    parts = []
    if with_q_tail:
        sc = layer.w_scale or {}
        parts.append(project(x[rows], layer.w_q, sc.get("q")))
    parts += [f["p_k"][rows], f["p_v"][rows]]
    tail[:, w - 1 - n_tail:] = np.concatenate(parts, axis=1).T
    return state, tail
