"""Pins for the oracle's parallel-branch Residual-DCN layer: a plain low-rank
cross net and an attention low-rank cross net with their own weights side by
side (section 'Residual DCN', second paragraph: 'paralleling a low-rank cross
net with an attention low-rank cross net'):

    t = U1 V1^T x_l + U2 (beta v2 + alpha softmax_j(q_i k_j / tau) v2) + b,
    x_{l+1} = x0 * t + x_l,   [v2; q; k] = [V2^T; Q^T; K^T] x_l.

Reductions checked: without the attention branch it is a textbook dense DCNv2
layer (numpy, W = U1 V1^T); without the plain branch it is the shared-weight
attention layer; with equal weights in both branches it is the shared layer
with the skip weight raised by one; with zero queries the attention is uniform
and the layer is dense with W = U1 V1^T + U2 (beta I + alpha/r 11^T) V2^T; the
two branches superpose linearly; the backward matches central differences.
"""
import numpy as np
import pytest

import oracle
from test_oracle_grad import fd_check


def weights(rng, L, d, r, scale=1.0):
    W = rng.standard_normal((L, 4 * r, d)) / np.sqrt(d) * 1.5 * scale
    U = rng.standard_normal((L, d, 2 * r)) / np.sqrt(2 * r)
    b = rng.standard_normal((L, d)) * 0.3
    return W, U, b


def dense_stack(x0, Ws, bs):
    x = x0.copy()
    for Wl, bl in zip(Ws, bs):
        x = x0 * (x @ Wl.T + bl) + x
    return x


def test_plain_branch_alone_is_dense_dcnv2():
    rng = np.random.default_rng(1)
    B, d, r, L = 5, 20, 6, 3
    x0 = rng.standard_normal((B, d))
    W, U, b = weights(rng, L, d, r)
    U[:, :, r:] = 0
    got = oracle.forward(x0, list(W), list(U), list(b), 1.0, 1.0, 1.0, parallel=True)
    ref = dense_stack(x0, [U[l, :, :r] @ W[l, :r] for l in range(L)], b)
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("alpha,beta,tau", [(1.0, 1.0, 1.0), (0.7, 0.3, 0.5)])
def test_attention_branch_alone_is_shared_layer(alpha, beta, tau):
    rng = np.random.default_rng(2)
    B, d, r, L = 4, 18, 5, 2
    x0 = rng.standard_normal((B, d))
    W, U, b = weights(rng, L, d, r)
    U[:, :, :r] = 0
    got = oracle.forward(x0, list(W), list(U), list(b), alpha, beta, tau, parallel=True)
    ref = oracle.forward(x0, list(W[:, r:]), list(U[:, :, r:]), list(b), alpha, beta, tau)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-13)


def test_equal_branches_raise_the_skip_weight_by_one():
    rng = np.random.default_rng(3)
    B, d, r, L = 3, 16, 4, 2
    x0 = rng.standard_normal((B, d))
    W, U, b = weights(rng, L, d, r)
    W[:, :r] = W[:, r:2 * r]          # V1 = V2
    U[:, :, :r] = U[:, :, r:]         # U1 = U2
    alpha, beta = 0.8, 0.4
    got = oracle.forward(x0, list(W), list(U), list(b), alpha, beta, 2.0, parallel=True)
    ref = oracle.forward(x0, list(W[:, r:]), list(U[:, :, r:]), list(b), alpha, beta + 1.0, 2.0)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-13)


def test_zero_queries_give_dense_uniform_layer():
    rng = np.random.default_rng(4)
    B, d, r, L = 4, 14, 5, 2
    alpha, beta = 0.9, 0.6
    x0 = rng.standard_normal((B, d))
    W, U, b = weights(rng, L, d, r)
    W[:, 2 * r:3 * r] = 0             # Q = 0
    M = beta * np.eye(r) + alpha / r * np.ones((r, r))
    Ws = [U[l, :, :r] @ W[l, :r] + U[l, :, r:] @ M @ W[l, r:2 * r] for l in range(L)]
    got = oracle.forward(x0, list(W), list(U), list(b), alpha, beta, 1.0, parallel=True)
    np.testing.assert_allclose(got, dense_stack(x0, Ws, b), rtol=1e-11, atol=1e-12)


def test_branches_superpose():
    rng = np.random.default_rng(5)
    B, d, r = 6, 12, 4
    x0 = rng.uniform(0.5, 1.5, (B, d)) * rng.choice([-1, 1], (B, d))  # no zeros: t = (x1 - x0) / x0
    W, U, b = weights(rng, 1, d, r)
    t = lambda Uv: (oracle.forward(x0, list(W), list(Uv), list(b), 1.0, 1.0, 1.0, parallel=True) - x0) / x0 - b[0]
    Ua, Ub = U.copy(), U.copy()
    Ua[:, :, r:] = 0
    Ub[:, :, :r] = 0
    np.testing.assert_allclose(t(U), t(Ua) + t(Ub), rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("alpha,beta,tau", [(1.0, 1.0, 1.0), (0.5, 0.0, 0.25), (1.0, 0.7, 4.0)])
def test_parallel_backward_matches_central_differences(alpha, beta, tau):
    rng = np.random.default_rng(6)
    B, d, r, L = 3, 20, 6, 2
    x0 = rng.standard_normal((B, d))
    W, U, b = weights(rng, L, d, r)
    G = rng.standard_normal((B, d))
    loss = lambda: float((G * oracle.forward(x0, list(W), list(U), list(b), alpha, beta, tau, parallel=True)).sum())
    gx0, gW, gU, gb = oracle.backward(x0, list(W), list(U), list(b), G, alpha, beta, tau, parallel=True)
    assert gW.shape == W.shape and gU.shape == U.shape
    for arr, g in ((x0, gx0), (W, gW), (U, gU), (b, gb)):
        assert fd_check(loss, arr, g) < 1e-6
