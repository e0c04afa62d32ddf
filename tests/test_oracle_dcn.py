"""Pins for the oracle's cross stack (section 'Residual DCN').

Each test checks the oracle against something it does not compute itself:
  - a textbook dense DCNv2 layer with a materialised W (the low-rank layer with
    W = U V^T must equal it; the attention term off),
  - the full-rank special case, trivial weights and the polynomial degree,
  - closed forms and invariants of the per-sample softmax attention
    (uniform limit, rows summing to one, two-token logistic form, shift
    invariance along the softmax axis, key/value permutation),
  - invariance under a consistent permutation of the r low-rank coordinates,
  - linearity in the two parallel branches (plain low-rank path and attention path).
"""
import numpy as np
import pytest

import oracle


def rand_stack(rng, d, r, L, attn, bias_std=0.3):
    n = 3 if attn else 1
    W = [rng.standard_normal((n * r, d)) / np.sqrt(d) for _ in range(L)]
    U = [rng.standard_normal((d, r)) / np.sqrt(r) for _ in range(L)]
    b = [rng.standard_normal(d) * bias_std for _ in range(L)]
    return W, U, b


def dense_dcn(x0, Ws, bs):
    """Textbook DCNv2 cross layers: x_{l+1} = x0 * (W_l x_l + b_l) + x_l (rows are samples)."""
    x = x0.copy()
    for W, b in zip(Ws, bs):
        x = x0 * (x @ W.T + b) + x
    return x


@pytest.mark.parametrize("beta", [1.0, 0.5])
def test_lowrank_equals_dense_dcnv2(beta):
    rng = np.random.default_rng(1)
    B, d, r, L = 6, 20, 5, 3
    x0 = rng.standard_normal((B, d))
    W, U, b = rand_stack(rng, d, r, L, attn=False)
    got = oracle.forward(x0, W, U, b, alpha=0.0, beta=beta)
    ref = dense_dcn(x0, [beta * Ul @ Wl for Wl, Ul in zip(W, U)], b)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_full_rank_identity_projection():
    rng = np.random.default_rng(2)
    B, d, L = 4, 9, 2
    x0 = rng.standard_normal((B, d))
    U = [rng.standard_normal((d, d)) / 3 for _ in range(L)]
    b = [rng.standard_normal(d) for _ in range(L)]
    got = oracle.forward(x0, [np.eye(d)] * L, U, b, alpha=0.0, beta=1.0)
    x = x0.copy()
    for Ul, bl in zip(U, b):
        x = x0 * (x @ Ul.T + bl) + x
    np.testing.assert_allclose(got, x, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("attn", [False, True])
def test_trivial_weights(attn):
    rng = np.random.default_rng(3)
    B, d, r = 5, 12, 4
    x0 = rng.standard_normal((B, d))
    W, _, _ = rand_stack(rng, d, r, 2, attn)
    alpha = 1.0 if attn else 0.0
    zeros_u = [np.zeros((d, r))] * 2
    # U = 0, b = 0: every layer is the identity
    np.testing.assert_array_equal(oracle.forward(x0, W, zeros_u, [np.zeros(d)] * 2, alpha, 1.0), x0)
    # U = 0, b = -1: x1 = -x0 + x0 = 0, then x2 = x0 * (-1) + 0
    np.testing.assert_array_equal(oracle.forward(x0, W[:1], zeros_u[:1], [-np.ones(d)], alpha, 1.0), 0 * x0)
    np.testing.assert_array_equal(oracle.forward(x0, W, zeros_u, [-np.ones(d)] * 2, alpha, 1.0), -x0)


def test_polynomial_degree():
    """alpha = 0, b = 0: x_L(lam * x0) is a polynomial in lam of degree L+1 with no constant term."""
    rng = np.random.default_rng(4)
    B, d, r, L = 3, 10, 4, 3
    x0 = rng.standard_normal((B, d))
    W, U, _ = rand_stack(rng, d, r, L, attn=False)
    zb = [np.zeros(d)] * L
    lams = np.arange(L + 3, dtype=np.float64) - 1.0
    ys = np.stack([oracle.forward(lam * x0, W, U, zb, 0.0, 1.0) for lam in lams])
    np.testing.assert_array_equal(ys[1], 0 * x0)  # lam = 0
    # (L+2)-th finite difference over unit steps vanishes for degree <= L+1 ...
    diff = ys.copy()
    for _ in range(L + 2):
        diff = diff[1:] - diff[:-1]
    scale = np.abs(ys).max()
    assert np.abs(diff).max() <= 1e-10 * scale
    # ... and the (L+1)-th does not (degree exactly L+1)
    diff = ys.copy()
    for _ in range(L + 1):
        diff = diff[1:] - diff[:-1]
    assert np.abs(diff).max() > 1e-3 * scale


def test_attention_rows_sum_to_one_and_constant_value():
    rng = np.random.default_rng(5)
    r = 16
    q, k = rng.standard_normal(r) * 3, rng.standard_normal(r) * 3
    A, o, h = oracle.attention(q, k, np.full(r, 2.5), alpha=1.0, beta=0.0, tau=0.7)
    np.testing.assert_allclose(A.sum(1), 1.0, rtol=1e-14)
    assert np.all(A > 0)
    np.testing.assert_allclose(o, 2.5, rtol=1e-14)
    np.testing.assert_allclose(h, 2.5, rtol=1e-14)


def test_attention_uniform_limits():
    rng = np.random.default_rng(6)
    r = 12
    q, k, v = (rng.standard_normal(r) for _ in range(3))
    for qq, kk, tau in ((np.zeros(r), k, 1.0), (q, np.zeros(r), 1.0), (q, k, 1e15)):
        A, o, h = oracle.attention(qq, kk, v, alpha=1.0, beta=1.0, tau=tau)
        np.testing.assert_allclose(A, 1.0 / r, rtol=1e-12)
        np.testing.assert_allclose(o, v.mean(), rtol=1e-12)
        np.testing.assert_allclose(h, v + v.mean(), rtol=1e-12)


@pytest.mark.parametrize("tau", [0.25, 1.0, 4.0])
def test_attention_two_tokens_logistic(tau):
    rng = np.random.default_rng(7)
    q, k, v = (rng.standard_normal(2) * 2 for _ in range(3))
    A, o, _ = oracle.attention(q, k, v, alpha=1.0, beta=0.0, tau=tau)
    p0 = 1.0 / (1.0 + np.exp(q * (k[1] - k[0]) / tau))
    np.testing.assert_allclose(A[:, 0], p0, rtol=1e-13)
    np.testing.assert_allclose(o, p0 * v[0] + (1 - p0) * v[1], rtol=1e-13)


def test_attention_single_token():
    A, o, h = oracle.attention([1.7], [-3.0], [0.4], alpha=2.0, beta=0.5, tau=1.0)
    assert A[0, 0] == 1.0 and o[0] == 0.4 and h[0] == pytest.approx(0.5 * 0.4 + 2.0 * 0.4)


def test_attention_softmax_axis_and_permutations():
    rng = np.random.default_rng(8)
    r = 10
    q, k, v = (rng.standard_normal(r) for _ in range(3))
    _, o, _ = oracle.attention(q, k, v, 1.0, 0.0, 1.3)
    # a constant added to every key shifts each row's scores by a constant: no change
    _, o2, _ = oracle.attention(q, k + 5.0, v, 1.0, 0.0, 1.3)
    np.testing.assert_allclose(o2, o, rtol=1e-12)
    # a constant added to every query is not such a shift
    _, o3, _ = oracle.attention(q + 5.0, k, v, 1.0, 0.0, 1.3)
    assert np.abs(o3 - o).max() > 1e-3
    # permuting the (key, value) tokens together leaves o unchanged; permuting queries permutes o
    p = rng.permutation(r)
    _, o4, _ = oracle.attention(q, k[p], v[p], 1.0, 0.0, 1.3)
    np.testing.assert_allclose(o4, o, rtol=1e-12)
    _, o5, _ = oracle.attention(q[p], k, v, 1.0, 0.0, 1.3)
    np.testing.assert_allclose(o5, o[p], rtol=1e-12)


@pytest.mark.parametrize("attn", [False, True])
def test_rank_permutation_invariance(attn):
    rng = np.random.default_rng(9)
    B, d, r, L = 4, 14, 6, 2
    x0 = rng.standard_normal((B, d))
    W, U, b = rand_stack(rng, d, r, L, attn)
    p = rng.permutation(r)
    n = 3 if attn else 1
    rows = np.concatenate([blk * r + p for blk in range(n)])
    Wp = [Wl[rows] for Wl in W]
    Up = [Ul[:, p] for Ul in U]
    alpha = 1.0 if attn else 0.0
    np.testing.assert_allclose(oracle.forward(x0, Wp, Up, b, alpha, 1.0),
                               oracle.forward(x0, W, U, b, alpha, 1.0), rtol=1e-12, atol=1e-12)


def test_uniform_attention_stack_equals_dense_dcn():
    """Query block zero => A = 11^T / r, so the layer is DCNv2 with W = U (beta I + alpha/r 11^T) V^T."""
    rng = np.random.default_rng(10)
    B, d, r, L = 5, 16, 4, 2
    x0 = rng.standard_normal((B, d))
    W, U, b = rand_stack(rng, d, r, L, attn=True)
    for Wl in W:
        Wl[r:2 * r] = 0.0
    alpha, beta = 0.7, 1.2
    M = beta * np.eye(r) + alpha / r * np.ones((r, r))
    ref = dense_dcn(x0, [Ul @ M @ Wl[:r] for Wl, Ul in zip(W, U)], b)
    np.testing.assert_allclose(oracle.forward(x0, W, U, b, alpha, beta), ref, rtol=1e-12, atol=1e-12)


def test_branches_add_linearly():
    """One layer: t = U(beta v + alpha o) + b, i.e. a plain low-rank branch plus an attention branch."""
    rng = np.random.default_rng(11)
    B, d, r = 4, 12, 5
    x0 = rng.standard_normal((B, d))
    W, U, b = rand_stack(rng, d, r, 1, attn=True)
    f = lambda a, bt: (oracle.forward(x0, W, U, b, a, bt) - x0) / x0 - b[0]  # = U h per sample
    np.testing.assert_allclose(f(1.0, 1.0), f(1.0, 0.0) + f(0.0, 1.0) * 1.0, rtol=1e-9, atol=1e-12)
