"""The chunked form of the Gated DeltaNet recurrence that the HIP scan kernel
evaluates, written here in fp64 numpy and checked against the oracle's
token-by-token recurrence (Section 2.1, Eq. recurrence).  This pins the
algebra the kernel relies on, independently of any GPU code.

Within a chunk of C rows that starts from state M0 (M = S^T, [d_k, d_v]), with
G_i = sum_{s<=i} log alpha_s:

    A_ij = beta_i exp(G_i - G_j) k_i.k_j   (i > j), else 0
    T    = (I + A)^{-1}
    U    = T diag(beta) V,    W = T diag(beta exp(G)) K
    Delta = U - W M0
    M_C  = exp(G_C) M0 + K^T diag(exp(G_C - G)) Delta

It follows from unrolling the recurrence over the chunk (Eq. unrolled): the
rank-one writes delta_i = beta_i (v_i - alpha_i S_{i-1} k_i) satisfy the
unit-lower-triangular system (I + A) Delta = diag(beta) V - diag(beta e^G) K M0.
"""
import numpy as np
import pytest

import oracle


def chunked_state(k, v, g, beta, C, M0=None):
    """k [L, dk] (unit rows), v [L, dv], g = log alpha [L], beta [L]."""
    L, dk = k.shape
    dv = v.shape[1]
    M = np.zeros((dk, dv)) if M0 is None else M0.copy()
    for c0 in range(0, L, C):
        K, V = k[c0:c0 + C], v[c0:c0 + C]
        gc, bc = g[c0:c0 + C], beta[c0:c0 + C]
        n = K.shape[0]
        G = np.cumsum(gc)
        lower = np.tri(n, n, -1, dtype=bool)
        dG = np.where(lower, G[:, None] - G[None, :], -np.inf)   # only i > j is used
        A = bc[:, None] * np.exp(dG) * (K @ K.T)
        T = np.linalg.inv(np.eye(n) + A)
        U = T @ (bc[:, None] * V)
        W = T @ ((bc * np.exp(G))[:, None] * K)
        Delta = U - W @ M
        M = np.exp(G[-1]) * M + K.T @ (np.exp(G[-1] - G)[:, None] * Delta)
    return M


def token_state(k, v, g, beta, M0=None):
    S0 = None if M0 is None else M0.T[None]
    S = oracle.gated_delta_recurrence(k[:, None, :], v[:, None, :], np.exp(g)[:, None], beta[:, None], S0)
    return S[0].T


@pytest.mark.parametrize("L", [1, 2, 3, 4, 5, 63, 64, 65, 127, 128, 200])
@pytest.mark.parametrize("C", [16, 32, 64])
def test_chunked_equals_token_recurrence(L, C):
    r = np.random.default_rng(L * 100 + C)
    dk, dv = 16, 8
    k = r.standard_normal((L, dk)); k /= np.linalg.norm(k, axis=1, keepdims=True)
    v = r.standard_normal((L, dv))
    g = -r.uniform(0.0, 3.0, L)
    beta = r.uniform(0, 1, L)
    M0 = r.standard_normal((dk, dv))
    for init in (None, M0):
        ref = token_state(k, v, g, beta, init)
        got = chunked_state(k, v, g, beta, C, init)
        assert np.linalg.norm(got - ref) <= 1e-12 * max(np.linalg.norm(ref), 1e-300)


def test_chunked_strong_decay_no_overflow():
    """Cumulative log-decay of -10^3 inside a chunk: only differences
    G_i - G_j <= 0 are exponentiated, so nothing overflows."""
    r = np.random.default_rng(9)
    L, dk, dv = 96, 8, 4
    k = r.standard_normal((L, dk)); k /= np.linalg.norm(k, axis=1, keepdims=True)
    v = r.standard_normal((L, dv))
    g = -r.uniform(10.0, 40.0, L)
    beta = r.uniform(0, 1, L)
    with np.errstate(over="raise", invalid="raise"):
        got = chunked_state(k, v, g, beta, 64)
    ref = token_state(k, v, g, beta)
    assert np.linalg.norm(got - ref) <= 1e-12 * np.linalg.norm(ref)


def test_padding_rows_are_inert():
    """Rows with k = v = 0, g = 0, beta = 0 appended to a partial chunk leave
    the state unchanged (the kernel pads the last chunk this way)."""
    r = np.random.default_rng(10)
    L, dk, dv = 70, 8, 4
    k = r.standard_normal((L, dk)); k /= np.linalg.norm(k, axis=1, keepdims=True)
    v = r.standard_normal((L, dv)); g = -r.uniform(0, 1, L); beta = r.uniform(0, 1, L)
    pad = 128 - L
    kp = np.concatenate([k, np.zeros((pad, dk))]); vp = np.concatenate([v, np.zeros((pad, dv))])
    gp = np.concatenate([g, np.zeros(pad)]); bp = np.concatenate([beta, np.zeros(pad)])
    np.testing.assert_allclose(chunked_state(kp, vp, gp, bp, 64), token_state(k, v, g, beta), rtol=1e-12, atol=1e-14)


def chunked_outputs(k, v, q, g, beta, C, M0=None):
    """Per-token outputs o_i = M_i^T q_i in chunk form.  Inside a chunk from
    M0 the state after row i is M_i = e^{G_i} M0 + sum_{j<=i} e^{G_i - G_j}
    k_j delta_j^T, so
        O = diag(e^G) Q M0 + (tril(Q K^T) * e^{G_i - G_j}) Delta
    with Delta = U - W M0 as for the state."""
    L, dk = k.shape
    dv = v.shape[1]
    M = np.zeros((dk, dv)) if M0 is None else M0.copy()
    O = np.zeros((L, dv))
    for c0 in range(0, L, C):
        K, V, Q = k[c0:c0 + C], v[c0:c0 + C], q[c0:c0 + C]
        gc, bc = g[c0:c0 + C], beta[c0:c0 + C]
        n = K.shape[0]
        G = np.cumsum(gc)
        lower = np.tri(n, n, -1, dtype=bool)
        dG = np.where(lower, G[:, None] - G[None, :], -np.inf)
        A = bc[:, None] * np.exp(dG) * (K @ K.T)
        T = np.linalg.inv(np.eye(n) + A)
        Delta = T @ (bc[:, None] * V) - T @ ((bc * np.exp(G))[:, None] * K) @ M
        causal = np.where(np.tri(n, n, 0, dtype=bool), np.exp(np.where(np.tri(n, n, 0, dtype=bool),
                                                                         G[:, None] - G[None, :], 0.0)), 0.0)
        O[c0:c0 + n] = np.exp(G)[:, None] * (Q @ M) + (causal * (Q @ K.T)) @ Delta
        M = np.exp(G[-1]) * M + K.T @ (np.exp(G[-1] - G)[:, None] * Delta)
    return O, M


@pytest.mark.parametrize("L", [1, 5, 63, 64, 65, 130])
@pytest.mark.parametrize("C", [32, 64])
def test_chunked_outputs_equal_token_outputs(L, C):
    """The output algebra of the group-replay kernel (chunk form) against the
    oracle's token-by-token read-out o_t = S_t q_t, with a non-zero start
    state; catches a strict instead of an inclusive causal mask."""
    from oracle import block
    r = np.random.default_rng(L * 7 + C)
    dk, dv = 16, 8
    k = r.standard_normal((L, dk)); k /= np.linalg.norm(k, axis=1, keepdims=True)
    q = r.standard_normal((L, dk)) * 0.3
    v = r.standard_normal((L, dv))
    g = -r.uniform(0.0, 3.0, L)
    beta = r.uniform(0, 1, L)
    M0 = r.standard_normal((dk, dv))
    O, M = chunked_outputs(k, v, q, g, beta, C, M0)
    S, O_ref = block.gated_delta_outputs(k[:, None], v[:, None], q[:, None], np.exp(g)[:, None], beta[:, None],
                                         M0.T[None])
    np.testing.assert_allclose(O, O_ref[:, 0], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(M, S[0].T, rtol=1e-10, atol=1e-12)
