"""Pins of the fp64 oracle against facts fixed outside the oracle itself:
library routines that define the same operation, closed forms, invariants of
the recurrence, the paper's unrolled form (Section 2.1, Eq. unrolled), and the
paper's printed storage sizes (Appendix A, Table 'Model parameters and the
resulting sizes').  Each test names the mistake it is there to catch."""
import json
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

import oracle
from oracle import crec
from workloads import Shape, LayerInputs, F32

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
rng0 = np.random.default_rng(1234)


# ---------------------------------------------------------------- projection
def test_project_matches_bruteforce_loops():
    """Catches a transposed weight or a dropped per-channel scale."""
    x = rng0.standard_normal((3, 5))
    w = rng0.standard_normal((4, 5))
    s = rng0.uniform(0.5, 2.0, 4)
    got = oracle.project(x, w, s)
    for t in range(3):
        for n in range(4):
            ref = sum(x[t, d] * w[n, d] * s[n] for d in range(5))
            assert abs(got[t, n] - ref) < 1e-13
    assert got.shape == (3, 4)


# ---------------------------------------------------------------------- conv
@pytest.mark.parametrize("L", [1, 2, 3, 4, 9])
def test_conv_matches_torch_conv1d(L):
    """Causal depthwise conv == torch conv1d(groups=C, padding=w-1) truncated
    to the first L outputs.  Catches a reversed tap order or an off-by-one lag."""
    C, w = 5, 4
    p = rng0.standard_normal((L, C))
    taps = rng0.standard_normal((C, w))
    ref = torch.nn.functional.conv1d(torch.from_numpy(p.T[None]), torch.from_numpy(taps[:, None, :]),
                                     padding=w - 1, groups=C)[0, :, :L].numpy().T
    np.testing.assert_allclose(oracle.causal_depthwise_conv(p, taps), ref, rtol=0, atol=1e-13)


def test_conv_matches_numpy_convolve():
    L, C, w = 11, 3, 4
    p = rng0.standard_normal((L, C))
    taps = rng0.standard_normal((C, w))
    y = oracle.causal_depthwise_conv(p, taps)
    for c in range(C):
        np.testing.assert_allclose(y[:, c], np.convolve(p[:, c], taps[c, ::-1])[:L], atol=1e-13)


def test_conv_current_row_tap_is_last():
    """Taps (0,..,0,1) leave the input unchanged; (1,0,..,0) delays it by w-1."""
    p = rng0.standard_normal((6, 2))
    ident = np.zeros((2, 4)); ident[:, 3] = 1
    np.testing.assert_array_equal(oracle.causal_depthwise_conv(p, ident), p)
    delay = np.zeros((2, 4)); delay[:, 0] = 1
    out = oracle.causal_depthwise_conv(p, delay)
    np.testing.assert_array_equal(out[3:], p[:3])
    np.testing.assert_array_equal(out[:3], 0)


# --------------------------------------------------------- activations/gates
def test_activations_match_library_routines():
    x = np.linspace(-60, 60, 2001)
    np.testing.assert_allclose(oracle.sigmoid(x), scipy.special.expit(x), rtol=1e-14, atol=1e-300)
    np.testing.assert_allclose(oracle.softplus(x), np.logaddexp(0.0, x), rtol=1e-14)
    np.testing.assert_allclose(oracle.silu(x), torch.nn.functional.silu(torch.from_numpy(x)).numpy(),
                               rtol=1e-14, atol=1e-300)
    assert oracle.silu(np.array([0.0]))[0] == 0.0


def test_gates_closed_forms():
    """softplus(0) = ln 2, so alpha = 2^-exp(A_log); A_log = ln 3 gives 1/8.
    Catches a missing exp on A_log, a sign error, or swapped a/b."""
    a = np.array([[0.0, -1.0]])
    b = np.array([[0.0, 2.0]])
    alpha, beta = oracle.decay_erase_gates(a, b, np.array([math.log(3.0), -np.inf]), np.array([0.0, 1.0]))
    assert abs(alpha[0, 0] - 0.125) < 1e-15
    assert alpha[0, 1] == 1.0               # A_log -> -inf: no decay
    assert beta[0, 0] == 0.5
    assert abs(beta[0, 1] - 1.0 / (1.0 + math.exp(-2.0))) < 1e-15
    _, beta_off = oracle.decay_erase_gates(a, np.array([[-np.inf, -800.0]]), np.zeros(2), np.zeros(2))
    assert np.all(beta_off == 0.0)          # b -> -inf: no erase/write
    al, _ = oracle.decay_erase_gates(np.array([[-1e4]]), np.array([[0.0]]), np.array([0.0]), np.array([0.0]))
    assert al[0, 0] == 1.0                   # softplus(-1e4) underflows to 0: alpha -> 1


def test_l2_normalize_norm_identity():
    """||k/sqrt(s+eps)||^2 = s/(s+eps) exactly (up to rounding)."""
    k = rng0.standard_normal((7, 3, 16)) * 0.01
    eps = 1e-6
    s = np.sum(k * k, axis=-1)
    kn = oracle.l2_normalize(k, eps)
    np.testing.assert_allclose(np.sum(kn * kn, axis=-1), s / (s + eps), rtol=1e-14)


def test_key_head_grouping():
    assert [oracle.key_head_of(h, 16, 32) for h in (0, 1, 2, 31)] == [0, 0, 1, 15]
    assert [oracle.key_head_of(h, 16, 48) for h in (0, 2, 3, 47)] == [0, 0, 1, 15]
    assert [oracle.key_head_of(h, 4, 4) for h in range(4)] == [0, 1, 2, 3]


# ----------------------------------------------------------------- recurrence
# Every recurrence pin runs on both implementations: the numpy loops and the
# plain-C twin (oracle/recurrence.c) that full-size parity tests use.
IMPLS = ["numpy", "c"]
if not crec.available():
    crec.build()


def _gdn(impl):
    return lambda *a: oracle.recurrence("gdn", *a, impl=impl)


def _decay(impl):
    return lambda *a: oracle.recurrence("decay", *a, impl=impl)


@pytest.mark.parametrize("kind", ["gdn", "decay"])
def test_c_twin_matches_numpy_recurrence(kind):
    """Implementation independence: the C twin and the numpy loops agree to
    1e-12 relative on random inputs with d_k != d_v, a non-zero initial state,
    unnormalised keys and several heads.  Catches a stride or orientation
    mistake in either."""
    for seed, (L, H, dk, dv) in enumerate([(1, 1, 3, 5), (37, 3, 8, 6), (130, 2, 32, 16)]):
        r = np.random.default_rng(100 + seed)
        k = r.standard_normal((L, H, dk)) * 0.4
        v = r.standard_normal((L, H, dv))
        alpha = r.uniform(0.2, 1.0, (L, H))
        beta = r.uniform(0.0, 1.0, (L, H))
        S0 = r.standard_normal((H, dv, dk))
        a = oracle.recurrence(kind, k, v, alpha, beta, S0, impl="numpy")
        b = oracle.recurrence(kind, k, v, alpha, beta, S0, impl="c")
        assert np.linalg.norm(a - b) <= 1e-12 * np.linalg.norm(a)
        assert np.array_equal(oracle.recurrence(kind, k[:0], v[:0], alpha[:0], beta[:0], S0, impl="c"), S0)

def _rand_inputs(L, H=2, dk=5, dv=3, unit=True, seed=0):
    r = np.random.default_rng(seed)
    k = r.standard_normal((L, H, dk))
    if unit:
        k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = r.standard_normal((L, H, dv))
    alpha = r.uniform(0.3, 1.0, (L, H))
    beta = r.uniform(0.0, 1.0, (L, H))
    return k, v, alpha, beta


@pytest.mark.parametrize("impl", IMPLS)
def test_recurrence_matches_paper_unrolled_form(impl):
    """Eq. (unrolled): S_n = sum_i Phi_{n,i}(B_i) with A_t(S) = S R_t,
    R_t = alpha_t (I - beta_t k_t k_t^T) and B_t = beta_t v_t k_t^T, evaluated as
    explicit matrix products.  Non-symmetric random data makes a transposed
    state, a wrong sign of the erase, or a missing decay fail."""
    L, H, dk, dv = 9, 2, 5, 3
    k, v, alpha, beta = _rand_inputs(L, H, dk, dv, unit=False)
    S = _gdn(impl)(k, v, alpha, beta)
    for h in range(H):
        R = [alpha[t, h] * (np.eye(dk) - beta[t, h] * np.outer(k[t, h], k[t, h])) for t in range(L)]
        total = np.zeros((dv, dk))
        for i in range(L):
            term = beta[i, h] * np.outer(v[i, h], k[i, h])
            for t in range(i + 1, L):
                term = term @ R[t]
            total += term
        np.testing.assert_allclose(S[h], total, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("impl", IMPLS)
def test_recurrence_identity_gates_keep_state(impl):
    """I1: alpha = 1, beta = 0 leaves any initial state unchanged."""
    k, v, _, _ = _rand_inputs(20)
    S0 = np.random.default_rng(3).standard_normal((2, 3, 5))
    S = _gdn(impl)(k, v, np.ones((20, 2)), np.zeros((20, 2)), S0)
    np.testing.assert_array_equal(S, S0)


@pytest.mark.parametrize("impl", IMPLS)
def test_recurrence_pure_decay(impl):
    """I2: beta = 0 gives S_L = prod(alpha) S_0."""
    k, v, alpha, _ = _rand_inputs(12)
    S0 = np.random.default_rng(4).standard_normal((2, 3, 5))
    S = _gdn(impl)(k, v, alpha, np.zeros((12, 2)), S0)
    np.testing.assert_allclose(S, np.prod(alpha, axis=0)[:, None, None] * S0, rtol=1e-14)


@pytest.mark.parametrize("impl", IMPLS)
def test_recurrence_exact_delta_write(impl):
    """I3: with beta_L = 1 and a unit key, S_L k_L = v_L whatever the history."""
    k, v, alpha, beta = _rand_inputs(15)
    beta[-1] = 1.0
    S0 = np.random.default_rng(5).standard_normal((2, 3, 5))
    S = _gdn(impl)(k, v, alpha, beta, S0)
    for h in range(2):
        np.testing.assert_allclose(S[h] @ k[-1, h], v[-1, h], rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("impl", IMPLS)
def test_recurrence_orthonormal_keys_store_last_value(impl):
    """I4: alpha = beta = 1 and keys from an orthonormal basis: the state is
    sum_e v_last(e) e^T (each write erases the previous value at its key)."""
    dk, dv, L = 4, 3, 11
    r = np.random.default_rng(6)
    basis = np.linalg.qr(r.standard_normal((dk, dk)))[0].T
    idx = r.integers(0, dk, L)
    k = basis[idx][:, None, :]
    v = r.standard_normal((L, 1, dv))
    S = _gdn(impl)(k, v, np.ones((L, 1)), np.ones((L, 1)))
    ref = np.zeros((dv, dk))
    for e in range(dk):
        hits = np.nonzero(idx == e)[0]
        if len(hits):
            ref += np.outer(v[hits[-1], 0], basis[e])
    np.testing.assert_allclose(S[0], ref, atol=1e-12)


@pytest.mark.parametrize("impl", IMPLS)
def test_recurrence_contraction_bound(impl):
    """I5 (the property suffix replay rests on, Section 1 and Section 2.1):
    ||S_L(S_0) - S_L(0)||_F <= ||S_0||_F prod(alpha) for unit keys, beta in [0,1]."""
    for seed in range(5):
        k, v, alpha, beta = _rand_inputs(40, H=3, dk=6, dv=4, seed=seed)
        S0 = np.random.default_rng(seed + 10).standard_normal((3, 4, 6)) * 5
        full = _gdn(impl)(k, v, alpha, beta, S0)
        replay = _gdn(impl)(k, v, alpha, beta)
        for h in range(3):
            lhs = np.linalg.norm(full[h] - replay[h])
            rhs = np.linalg.norm(S0[h]) * np.prod(alpha[:, h])
            assert lhs <= rhs * (1 + 1e-12) + 1e-300


@pytest.mark.parametrize("impl", IMPLS)
def test_recurrence_single_token_closed_form(impl):
    """I6: L = 1 from zero: S_1 = beta v k^T (catches an outer product in the
    wrong order)."""
    k, v, alpha, beta = _rand_inputs(1, unit=False)
    S = _gdn(impl)(k, v, alpha, beta)
    for h in range(2):
        np.testing.assert_allclose(S[h], beta[0, h] * np.outer(v[0, h], k[0, h]), rtol=1e-15)


@pytest.mark.parametrize("impl", IMPLS)
def test_recurrence_linear_in_values(impl):
    """I7: from zero, f(v + c v') = f(v) + c f(v') for fixed k, alpha, beta."""
    k, v, alpha, beta = _rand_inputs(17)
    v2 = np.random.default_rng(8).standard_normal(v.shape)
    lhs = _gdn(impl)(k, v + 2.5 * v2, alpha, beta)
    rhs = _gdn(impl)(k, v, alpha, beta) + 2.5 * _gdn(impl)(k, v2, alpha, beta)
    np.testing.assert_allclose(lhs, rhs, rtol=1e-12, atol=1e-13)


# ---------------------------------------------------------- whole-layer replay
def _tiny_layer(shape, T, seed=0):
    r = np.random.default_rng(seed)
    D, qk, vv, hv = shape.d_model, shape.n_k_heads * shape.d_k, shape.n_v_heads * shape.d_v, shape.n_v_heads
    n = lambda *s: r.standard_normal(s) * 0.3
    return LayerInputs(anchors=r.standard_normal((T, D)), w_q=n(qk, D), w_k=n(qk, D), w_v=n(vv, D),
                       w_a=n(hv, D), w_b=n(hv, D), conv_w=n(shape.c_kv, shape.conv_width),
                       a_log=r.uniform(0, 1, hv), dt_bias=r.standard_normal(hv))


def test_replay_single_row_closed_form():
    """L = 1: only the current-row tap sees data, so state = beta k_hat v^T in
    the [H_v][d_k][d_v] layout with k_hat = normalised silu(tap_last * W_k x)."""
    shape = Shape(6, 1, 2, 3, 2, anchor_dtype=F32, weight_dtype=F32, conv_dtype=F32, tail_dtype=F32)
    lay = _tiny_layer(shape, 1)
    x = lay.anchors
    state, tail = oracle.replay_segment(shape, lay, x)
    pk = x[0] @ lay.w_k.T
    pv = x[0] @ lay.w_v.T
    k = pk * lay.conv_w[:3, 3]
    k = k / (1 + np.exp(-k))
    k = k / np.sqrt(k @ k + shape.l2_eps)
    v = pv * lay.conv_w[3:, 3]
    v = v / (1 + np.exp(-v))
    b = 1 / (1 + np.exp(-(x[0] @ lay.w_b.T)))
    for h in range(2):
        np.testing.assert_allclose(state[h], b[h] * np.outer(k, v[2 * h:2 * h + 2]), rtol=1e-12)
    # tail: only the newest position holds data
    np.testing.assert_array_equal(tail[:, :2], 0)
    np.testing.assert_allclose(tail[:, 2], np.concatenate([x[0] @ lay.w_q.T, pk, pv]), rtol=1e-13)


@pytest.mark.parametrize("L", [0, 1, 2, 3, 5])
def test_replay_tail_is_raw_last_rows(L):
    shape = Shape(8, 2, 2, 4, 4, anchor_dtype=F32, weight_dtype=F32, conv_dtype=F32, tail_dtype=F32)
    lay = _tiny_layer(shape, max(L, 1), seed=L)
    x = lay.anchors[:L]
    state, tail = oracle.replay_segment(shape, lay, x)
    assert tail.shape == (shape.c_tail, 3)
    W = np.concatenate([lay.w_q, lay.w_k, lay.w_v])
    for j in range(3):
        t = L - 3 + j
        if t < 0:
            assert np.all(tail[:, j] == 0)
        else:
            np.testing.assert_allclose(tail[:, j], W @ x[t], rtol=1e-13)
    if L == 0:
        assert np.all(state == 0)


def test_replay_value_head_permutation():
    """I10: permuting value heads (W_v rows, W_a/W_b rows, A_log, dt_bias and
    v conv taps together) permutes the state; catches a value head reading the
    wrong gate row."""
    shape = Shape(8, 2, 2, 4, 4, anchor_dtype=F32, weight_dtype=F32, conv_dtype=F32, tail_dtype=F32)
    lay = _tiny_layer(shape, 10, seed=2)
    s1, _ = oracle.replay_segment(shape, lay, lay.anchors)
    perm = [1, 0]
    lay2 = _tiny_layer(shape, 10, seed=2)
    # keep keys: swap value heads only when both heads read distinct key heads
    # -> swap key heads as well so that head h keeps its key
    lay2.w_k = np.concatenate([lay.w_k[4:], lay.w_k[:4]])
    lay2.w_q = np.concatenate([lay.w_q[4:], lay.w_q[:4]])
    lay2.w_v = np.concatenate([lay.w_v[4:], lay.w_v[:4]])
    lay2.w_a = lay.w_a[perm]
    lay2.w_b = lay.w_b[perm]
    lay2.a_log = lay.a_log[perm]
    lay2.dt_bias = lay.dt_bias[perm]
    cw = lay.conv_w
    lay2.conv_w = np.concatenate([cw[4:8], cw[0:4], cw[12:16], cw[8:12]])
    s2, _ = oracle.replay_segment(shape, lay2, lay.anchors)
    np.testing.assert_allclose(s2, s1[perm], rtol=1e-12)


def test_replay_gqa_heads_share_key():
    """H_v = 2 H_k: value heads 0 and 1 read key head 0.  With identical gate
    and value weights for heads 0 and 1 their states must be identical, and
    differ from head 2 (key head 1)."""
    shape = Shape(8, 2, 4, 4, 4, anchor_dtype=F32, weight_dtype=F32, conv_dtype=F32, tail_dtype=F32)
    lay = _tiny_layer(shape, 12, seed=4)
    lay.w_v[4:8] = lay.w_v[0:4]
    lay.w_a[1] = lay.w_a[0]; lay.w_b[1] = lay.w_b[0]
    lay.a_log[1] = lay.a_log[0]; lay.dt_bias[1] = lay.dt_bias[0]
    lay.conv_w[8 + 4:8 + 8] = lay.conv_w[8:8 + 4]
    s, _ = oracle.replay_segment(shape, lay, lay.anchors)
    np.testing.assert_array_equal(s[0], s[1])
    assert np.abs(s[0] - s[2]).max() > 1e-6


def test_state_and_conv_sizes_match_paper_table():
    """Appendix A: B_rec = H_v d_k d_v * 4 (fp32 state), B_conv = C (w-1) * 2
    (bf16 conv state) with C = 2 H_k d_k + H_v d_v.  The oracle's output
    arrays for these three model shapes must hold exactly those element
    counts, and the checkpoint/naive per-token sizes follow."""
    tab = json.load(open(os.path.join(GOLDEN, "storage_table6.json")))
    w = tab["conv_width"]
    for name, m in tab["models"].items():
        shape = Shape(m["d"], m["H_k"], m["H_v"], m["d_k"], m["d_v"], conv_width=w)
        assert shape.c_tail == m["C"], name
        state = np.zeros((shape.n_v_heads, shape.d_k, shape.d_v), dtype=np.float32)
        tail = np.zeros((shape.c_tail, w - 1), dtype=np.float16)   # 2-byte storage
        assert state.nbytes == m["B_rec"], name
        assert tail.nbytes == m["B_conv"], name
        assert m["L_lin"] * (m["B_rec"] + m["B_conv"]) == m["B_ckpt"], name
        assert m["B_ckpt"] / 8192 == m["B_native_8192"], name
        assert m["L_lin"] * m["d"] * 2 == m["B_naive"], name


# ------------------------------------------------- per-head decay (Mamba2)
@pytest.mark.parametrize("impl", IMPLS)
def test_decay_recurrence_equals_gdn_for_orthogonal_keys(impl):
    """With mutually orthogonal unit keys the erase term S_{t-1} k_t vanishes
    (every earlier write is along an orthogonal key), so Gated DeltaNet and
    the decay-only recurrence give the same state.  Catches a decay applied
    to the write, a missing beta, or a transposed outer product."""
    rng = np.random.default_rng(21)
    L, H, dk, dv = 6, 2, 8, 5
    q, _ = np.linalg.qr(rng.standard_normal((dk, dk)))
    k = np.stack([q[:L].copy() for _ in range(H)], axis=1)          # [L, H, dk], orthonormal rows
    v = rng.standard_normal((L, H, dv))
    alpha = rng.uniform(0.5, 1.0, (L, H))
    beta = rng.uniform(0.1, 0.9, (L, H))
    S0 = rng.standard_normal((H, dv, dk)) @ np.diag([0.0] * dk)     # zero start
    assert np.allclose(_decay(impl)(k, v, alpha, beta, S0),
                       _gdn(impl)(k, v, alpha, beta, S0), atol=1e-12)


@pytest.mark.parametrize("impl", IMPLS)
def test_decay_recurrence_matches_the_unrolled_sum(impl):
    """The paper's unrolled form (Section 2.1, Eq. unrolled) with a scalar
    decay per head: S_n = prod(alpha) S_0 + sum_i (prod_{s>i} alpha_s) beta_i
    v_i k_i^T, evaluated as one weighted matrix product.  Catches an
    off-by-one in which decays a write receives."""
    rng = np.random.default_rng(22)
    L, H, dk, dv = 9, 3, 4, 6
    k = rng.standard_normal((L, H, dk))
    v = rng.standard_normal((L, H, dv))
    alpha = rng.uniform(0.3, 1.0, (L, H))
    beta = rng.uniform(0.1, 0.9, (L, H))
    S0 = rng.standard_normal((H, dv, dk))
    got = _decay(impl)(k, v, alpha, beta, S0)
    for h in range(H):
        w = np.array([np.prod(alpha[i + 1:, h]) * beta[i, h] for i in range(L)])
        want = np.prod(alpha[:, h]) * S0[h] + v[:, h].T @ np.diag(w) @ k[:, h]
        assert np.allclose(got[h], want, atol=1e-12)
