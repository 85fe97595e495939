"""Derive the dt_bias mean of the long-memory ("stress64") workload.

The workload skews the decay gates toward slow forgetting: dt_bias is drawn
as mu + 0.5 z, and mu is chosen so that the empirical mean of
alpha = exp(-exp(A_log) softplus(a + dt_bias)) over every (row, value head) of
the generated inputs is 0.995.  Gate values come from the oracle only.
Prints mu; the result is stored as workloads.LONG_MEMORY_DT_BIAS_MEAN.

    python tests/golden/derive_long_memory_dt_bias.py
"""
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))
import oracle  # noqa: E402
import workloads as W  # noqa: E402

TARGET = 0.995


def gate_inputs(rows=None, block=16384):
    """Decay-gate projections a = W_a h for the first ``rows`` anchor rows
    (all rows when None), streamed in blocks of the one anchor stream."""
    seed, shape, seg, _, _ = W._config_table("stress64")
    T = sum(seg) if rows is None else rows
    w_a = W.round_to_bf16(W.tensor_rng(seed, 0, "a").standard_normal(
        (shape.n_v_heads, shape.d_model), dtype=np.float32) * np.float32(0.02))
    g = W.tensor_rng(seed, 0, "anchors")
    parts = []
    for i in range(0, T, block):
        x = W.round_to_bf16(g.standard_normal((min(block, T - i), shape.d_model), dtype=np.float32))
        parts.append(oracle.project(x, w_a))
    a_log = W.tensor_rng(seed, 0, "a_log").uniform(np.log(1.0), np.log(16.0), size=shape.n_v_heads).astype(np.float32)
    z = W.tensor_rng(seed, 0, "dt_bias").standard_normal(shape.n_v_heads, dtype=np.float32)
    return np.concatenate(parts), z, a_log


def mean_alpha(a, z, a_log, mu):
    dt_bias = (np.float32(mu) + np.float32(0.5) * z).astype(np.float32)
    alpha, _ = oracle.decay_erase_gates(a, np.zeros_like(a), a_log, dt_bias)
    return float(alpha.mean())


def main():
    a, z, a_log = gate_inputs()
    lo, hi = -40.0, 0.0             # mean alpha rises as mu falls
    for _ in range(50):
        mid = 0.5 * (lo + hi)
        if mean_alpha(a, z, a_log, mid) > TARGET:
            lo = mid
        else:
            hi = mid
    mu = round(0.5 * (lo + hi), 3)
    print(f"mu = {mu}  mean alpha = {mean_alpha(a, z, a_log, mu):.6f}")


if __name__ == "__main__":
    main()
