"""Checks of the seeded input generator: storage-format rounding agrees with
torch's own bf16 / float8_e4m3fn casts (so the GPU path receives exactly the
values the oracle reads), draws are reproducible, and the named workloads have
the shapes they claim."""
import numpy as np
import pytest
import torch

import workloads as W


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 3
    ours = W.round_to_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(ours, ref)


def test_e4m3_rounding_matches_torch():
    r = np.random.default_rng(1)
    x = np.concatenate([r.uniform(-448, 448, 50000), r.standard_normal(50000) * 0.01,
                        r.standard_normal(50000)]).astype(np.float32)
    ours = W.round_to_e4m3(x)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).to(torch.float32).numpy()
    np.testing.assert_array_equal(ours, ref)


def test_e4m3_known_codes():
    """OCP E4M3 values: max normal 448, min normal 2^-6, min subnormal 2^-9."""
    vals = np.array([448.0, 2.0 ** -6, 2.0 ** -9, 1.0, 1.125, 0.0, 500.0, 2.0 ** -11])
    np.testing.assert_array_equal(W.round_to_e4m3(vals), [448.0, 2.0 ** -6, 2.0 ** -9, 1.0, 1.125, 0.0, 448.0, 0.0])


def test_fp8_quantisation_is_exact_in_storage():
    r = np.random.default_rng(2)
    w = r.standard_normal((64, 96)).astype(np.float32) * 0.02
    q, s = W.quantize_rows_e4m3(w)
    assert np.all(np.abs(q) <= 448)
    np.testing.assert_array_equal(torch.from_numpy(q).to(torch.float8_e4m3fn).to(torch.float32).numpy(), q)
    np.testing.assert_array_equal(torch.from_numpy(s).to(torch.bfloat16).to(torch.float32).numpy(), s)
    assert np.max(np.abs(q * s[:, None] - w) / np.max(np.abs(w))) < 0.07


def test_generator_is_seeded():
    shape = W.Shape(64, 2, 4, 16, 16)
    a = W.make_workload("x", shape, [5, 70], n_layers=2, seed=7)
    b = W.make_workload("x", shape, [5, 70], n_layers=2, seed=7)
    for la, lb in zip(a.layers, b.layers):
        np.testing.assert_array_equal(la.anchors, lb.anchors)
        np.testing.assert_array_equal(la.w_v, lb.w_v)
        np.testing.assert_array_equal(la.dt_bias, lb.dt_bias)
    np.testing.assert_array_equal(a.cu_seqlens, [0, 5, 75])


@pytest.mark.parametrize("name", W.CONFIG_NAMES)
def test_named_config_shapes(name):
    shape, seg, n_layers = W.config_shape(name)
    assert all(L % 64 == 0 for L in seg)
    if name == "tiny":
        assert (shape.d_model, shape.n_v_heads, shape.d_k, seg, n_layers) == (128, 2, 32, [256], 1)
    if name == "varlen16":
        assert len(seg) == 16 and all(512 <= L <= 4096 for L in seg)
        assert (shape.d_model, shape.n_k_heads, shape.n_v_heads) == (2560, 16, 32)
    if name == "stress64":
        assert len(seg) == 64 and all(1024 <= L <= 8192 for L in seg)
    if name == "multilayer12":
        assert n_layers == 12 and seg == [4096] * 4 and shape.weight_dtype == W.FP8


def test_tiny_config_values():
    wl = W.make_config("tiny")
    lay = wl.layers[0]
    assert lay.anchors.shape == (256, 128)
    assert abs(lay.w_k.std() - 0.02) < 0.002
    assert np.all((lay.a_log >= 0) & (lay.a_log <= np.log(16)))


def test_long_memory_gates_mean_alpha():
    """stress64 skews decay toward slow forgetting: mean alpha 0.995 over all
    rows (derived by tests/golden/derive_long_memory_dt_bias.py); a prefix of
    32768 rows must already sit within 5e-4 of it."""
    import importlib.util, os
    path = os.path.join(os.path.dirname(__file__), "golden", "derive_long_memory_dt_bias.py")
    spec = importlib.util.spec_from_file_location("derive_mu", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    a, z, a_log = mod.gate_inputs(rows=32768)
    m = mod.mean_alpha(a, z, a_log, W.LONG_MEMORY_DT_BIAS_MEAN)
    assert abs(m - 0.995) < 5e-4, m
