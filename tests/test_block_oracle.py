"""Pins of the group-replay oracle (oracle/block.py) against facts fixed
outside it: library routines for RMSNorm and SiLU, the paper's unrolled form
(Section 2.1, Eq. unrolled) for the per-token outputs, closed forms, residual
identities, and the already-pinned single-layer oracle for the mixer's state
and conv tail.  Each test names the mistake it would catch."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import block, crec
from workloads import F32, LayerInputs, Shape
from workloads.group import BlockInputs

if not crec.available():
    crec.build()

rng0 = np.random.default_rng(77)


def test_rms_norm_matches_torch():
    """Catches a missing mean (sum instead), eps outside the root, or a
    forgotten weight."""
    x = rng0.standard_normal((5, 12)) * 3
    w = rng0.uniform(0.5, 1.5, 12)
    ref = F.rms_norm(torch.from_numpy(x), (12,), torch.from_numpy(w), eps=1e-6).numpy()
    np.testing.assert_allclose(block.rms_norm(x, w, 1e-6), ref, rtol=1e-14)


def test_gated_rms_norm_matches_torch_composition():
    """Per value head norm over d_v with a shared weight, times SiLU(z).
    Catches a norm over all heads at once or a gate without SiLU."""
    L, H, dv = 4, 3, 8
    o = rng0.standard_normal((L, H, dv))
    z = rng0.standard_normal((L, H * dv))
    w = rng0.uniform(0.5, 1.5, dv)
    ref = (F.rms_norm(torch.from_numpy(o), (dv,), torch.from_numpy(w), eps=1e-6)
           * F.silu(torch.from_numpy(z).reshape(L, H, dv))).reshape(L, H * dv).numpy()
    np.testing.assert_allclose(block.gated_rms_norm(o, z, w, 1e-6), ref, rtol=1e-13)


def test_swiglu_mlp_bruteforce():
    """Catches gate and up swapped (SiLU on the wrong branch) or a transposed
    weight."""
    D, I = 5, 7
    u = rng0.standard_normal((2, D))
    wg, wu, wd = rng0.standard_normal((I, D)), rng0.standard_normal((I, D)), rng0.standard_normal((D, I))
    got = block.swiglu_mlp(u, wg, wu, wd)
    for t in range(2):
        hidden = []
        for i in range(I):
            g = sum(wg[i, d] * u[t, d] for d in range(D))
            up = sum(wu[i, d] * u[t, d] for d in range(D))
            hidden.append(g / (1 + np.exp(-g)) * up)
        for d in range(D):
            assert abs(got[t, d] - sum(wd[d, i] * hidden[i] for i in range(I))) < 1e-12


def _rand(L, H=2, dk=5, dv=3, seed=0):
    r = np.random.default_rng(seed)
    k = r.standard_normal((L, H, dk))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    q = r.standard_normal((L, H, dk))
    v = r.standard_normal((L, H, dv))
    return k, v, q, r.uniform(0.3, 1.0, (L, H)), r.uniform(0.0, 1.0, (L, H))


@pytest.mark.parametrize("impl", ["numpy", "c"])
def test_outputs_match_paper_unrolled_form(impl):
    """o_t = S_t q_t with S_t from Eq. (unrolled) as explicit matrix products:
    S_t = sum_{i<=t} beta_i v_i k_i^T R_{i+1} ... R_t, R = alpha (I - beta k k^T).
    Catches reading the state before the token's own write, or q and k
    swapped."""
    L, H, dk, dv = 7, 2, 5, 3
    k, v, q, alpha, beta = _rand(L, H, dk, dv)
    S, O = block.outputs_recurrence(k, v, q, alpha, beta, impl=impl)
    for h in range(H):
        R = [alpha[t, h] * (np.eye(dk) - beta[t, h] * np.outer(k[t, h], k[t, h])) for t in range(L)]
        for t in range(L):
            St = np.zeros((dv, dk))
            for i in range(t + 1):
                term = beta[i, h] * np.outer(v[i, h], k[i, h])
                for s in range(i + 1, t + 1):
                    term = term @ R[s]
                St += term
            np.testing.assert_allclose(O[t, h], St @ q[t, h], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(S, oracle.gated_delta_recurrence(k, v, alpha, beta), rtol=1e-12, atol=1e-13)


def test_outputs_single_token_and_twin_agreement():
    """L = 1 from zero: o_1 = beta (k . q) v (catches an outer product in the
    wrong order); the C twin equals the numpy loop to 1e-12."""
    k, v, q, alpha, beta = _rand(1, seed=3)
    _, O = block.gated_delta_outputs(k, v, q, alpha, beta)
    for h in range(2):
        np.testing.assert_allclose(O[0, h], beta[0, h] * (k[0, h] @ q[0, h]) * v[0, h], rtol=1e-14)
    k, v, q, alpha, beta = _rand(90, H=3, dk=16, dv=8, seed=4)
    S0 = np.random.default_rng(5).standard_normal((3, 8, 16))
    a = block.outputs_recurrence(k, v, q, alpha, beta, S0, impl="numpy")
    b = block.outputs_recurrence(k, v, q, alpha, beta, S0, impl="c")
    for x, y in zip(a, b):
        assert np.linalg.norm(x - y) <= 1e-12 * np.linalg.norm(x)


def _tiny_block(shape, T, d_ff=6, seed=0, zero_o=False, zero_down=False):
    r = np.random.default_rng(seed)
    D, qk, vv, hv = shape.d_model, shape.n_k_heads * shape.d_k, shape.n_v_heads * shape.d_v, shape.n_v_heads
    n = lambda *s: r.standard_normal(s) * 0.3
    mixer = LayerInputs(anchors=r.standard_normal((T, D)), w_q=n(qk, D), w_k=n(qk, D), w_v=n(vv, D), w_a=n(hv, D),
                        w_b=n(hv, D), conv_w=n(shape.c_kv, shape.conv_width), a_log=r.uniform(0, 1, hv),
                        dt_bias=r.standard_normal(hv))
    return BlockInputs(mixer=mixer, conv_q=n(qk, shape.conv_width), w_z=n(vv, D), norm_o=r.uniform(0.5, 1.5, shape.d_v),
                       w_o=np.zeros((D, vv)) if zero_o else n(D, vv), ln_in=r.uniform(0.5, 1.5, D),
                       ln_post=r.uniform(0.5, 1.5, D), w_gate=n(d_ff, D), w_up=n(d_ff, D),
                       w_down=np.zeros((D, d_ff)) if zero_down else n(D, d_ff))


SHAPE = Shape(8, 2, 4, 4, 4, anchor_dtype=F32, weight_dtype=F32, conv_dtype=F32, tail_dtype=F32)


def test_mixer_state_and_tail_equal_the_single_layer_oracle():
    """The mixer's state and conv tail on normalised inputs are exactly the
    single-layer replay (pinned separately) of the same rows: the query path
    must not disturb them.  Catches a q/k channel mix-up in the tail."""
    blk = _tiny_block(SHAPE, 11)
    x = block.rms_norm(blk.mixer.anchors, blk.ln_in, 1e-6)
    state, tail, O, z = block.gdn_mixer(SHAPE, blk, x)
    ref_state, ref_tail = oracle.replay_segment(SHAPE, blk.mixer, x)
    np.testing.assert_allclose(state, ref_state, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(tail, ref_tail, rtol=1e-13)
    assert O.shape == (11, 4, 4) and z.shape == (11, 16)


def test_mixer_query_path_single_row():
    """L = 1: q_hat = normalised SiLU(tap_last * W_q x) / sqrt(d_k), so
    o = beta (k_hat . q_hat) v per value head with its key head's q.  Catches
    a missing 1/sqrt(d_k) or the wrong conv tap on q."""
    blk = _tiny_block(SHAPE, 1, seed=2)
    x = blk.mixer.anchors
    _, _, O, _ = block.gdn_mixer(SHAPE, blk, x)
    f = oracle.layer_features(SHAPE, blk.mixer, x)
    q = x[0] @ blk.mixer.w_q.T * blk.conv_q[:, 3]
    q = q / (1 + np.exp(-q))
    q = q.reshape(2, 4)
    q = q / np.sqrt(np.sum(q * q, axis=1, keepdims=True) + SHAPE.l2_eps) / 2.0
    for h in range(4):
        kh = h // 2
        want = f["beta"][0, h] * (f["k"][0, kh] @ q[kh]) * f["v"][0, h]
        np.testing.assert_allclose(O[0, h], want, rtol=1e-12)


def test_block_residual_identities():
    """With W_o = 0 and W_down = 0 the block is the identity (pre-norm
    residuals); with W_down = 0 only, h_next - h is exactly W_o y.  Catches a
    norm applied to the residual stream or a dropped residual."""
    blk = _tiny_block(SHAPE, 9, seed=5, zero_o=True, zero_down=True)
    h = blk.mixer.anchors
    h_next, _, _, _ = block.block_forward(SHAPE, blk, h)
    np.testing.assert_array_equal(h_next, h)
    blk = _tiny_block(SHAPE, 9, seed=5, zero_down=True)
    h_next, _, _, y = block.block_forward(SHAPE, blk, h)
    np.testing.assert_allclose(h_next - h, y @ blk.w_o.T, rtol=1e-12, atol=1e-14)


def test_group_chains_block_outputs():
    """Layer j + 1 of a group replays from layer j's block output: its state
    equals the single-layer oracle on RMSNorm(block output).  Catches
    replaying every layer from the group-entry anchor."""
    blocks = [_tiny_block(SHAPE, 13, seed=s) for s in (7, 8, 9)]
    x = blocks[0].mixer.anchors
    res, inputs = block.replay_group_segment(SHAPE, blocks, x)
    h = x
    for j, blk in enumerate(blocks):
        np.testing.assert_allclose(inputs[j], h, rtol=1e-13)
        xs = block.rms_norm(h, blk.ln_in, 1e-6)
        ref_state, _ = oracle.replay_segment(SHAPE, blk.mixer, xs)
        np.testing.assert_allclose(res[j][0], ref_state, rtol=1e-11, atol=1e-13)
        h, _, _, _ = block.block_forward(SHAPE, blk, h)
    assert not np.allclose(res[1][0], oracle.replay_segment(SHAPE, blocks[1].mixer,
                                                            block.rms_norm(x, blocks[1].ln_in, 1e-6))[0])
