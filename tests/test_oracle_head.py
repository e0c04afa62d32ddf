"""Pins of the head oracle (gated MLP, logit, isotonic calibration, log loss).

Each pin checks the oracle against something other than itself: a library
routine (torch float64 layers, autograd, binary cross-entropy, searchsorted),
central finite differences, closed forms the calibration equation reduces to,
its isotonic property, continuity, and its integral form by brute force.
"""
import numpy as np
import pytest
import torch

from oracle import head as H


def _params(rng, widths, gated, K, d_in):
    W, b, G, c = [], [], [], []
    prev = d_in
    for n in widths:
        W.append(rng.standard_normal((n, prev)) / np.sqrt(prev))
        b.append(0.1 * rng.standard_normal(n))
        G.append(rng.standard_normal(prev) / np.sqrt(prev))
        c.append(0.3 * rng.standard_normal())
        prev = n
    p = {"W": W, "b": b, "w_out": rng.standard_normal(prev) / np.sqrt(prev), "b_out": 0.2,
         "cal_w": 0.5 + rng.random(K), "cal_b": -0.3, "lo": -2.0, "step": 0.5}
    if gated:
        p["G"], p["c"] = G, c
    return p


# ---------------------------------------------------------------------------
# MLP
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("gated", [False, True])
def test_mlp_forward_matches_torch_layers(gated):
    rng = np.random.default_rng(1)
    p = _params(rng, [12, 9, 7], gated, 4, 10)
    x = rng.standard_normal((6, 10))
    a, s = H.mlp_forward(x, p["W"], p["b"], p.get("G"), p.get("c"))
    t = torch.from_numpy(x)
    for l in range(3):
        lin = torch.nn.functional.linear(t, torch.from_numpy(p["W"][l]), torch.from_numpy(p["b"][l]))
        out = torch.relu(lin)
        if gated:
            gl = torch.nn.functional.linear(t, torch.from_numpy(p["G"][l])[None, :], torch.tensor([p["c"][l]], dtype=torch.float64))
            out = out * torch.sigmoid(gl)
        t = out
        np.testing.assert_allclose(a[l + 1], t.numpy(), rtol=1e-13, atol=1e-14)
    assert len(s) == (3 if gated else 0)


def test_gate_reads_the_layer_input():
    """Worked example: x = (1, 2), W = 2I, b = 0, g = (1, -1), c = 0.5. The gate logit
    is g.x + c = -0.5 (from the input; the layer output (2, 4) would give -1.5)."""
    x = np.array([[1.0, 2.0]])
    a, s = H.mlp_forward(x, [2 * np.eye(2)], [np.zeros(2)], [np.array([1.0, -1.0])], [0.5])
    assert s[0][0] == pytest.approx(-0.5)
    sig = 1.0 / (1.0 + np.exp(0.5))
    np.testing.assert_allclose(a[1][0], [2 * sig, 4 * sig], rtol=1e-15)


def test_constant_gate_scales_the_plain_layer():
    rng = np.random.default_rng(2)
    p = _params(rng, [8], True, 2, 5)
    x = rng.standard_normal((4, 5))
    plain, _ = H.mlp_forward(x, p["W"], p["b"])
    gated, _ = H.mlp_forward(x, p["W"], p["b"], [np.zeros(5)], [0.0])
    np.testing.assert_allclose(gated[1], 0.5 * plain[1], rtol=1e-15)


def test_identity_layers_are_relu():
    x = np.array([[1.5, -2.0, 0.0, 3.0]])
    a, _ = H.mlp_forward(x, [np.eye(4), np.eye(4)], [np.zeros(4), np.zeros(4)])
    np.testing.assert_array_equal(a[2], np.maximum(x, 0))


def test_ungated_bias_free_mlp_is_positively_homogeneous():
    rng = np.random.default_rng(3)
    W = [rng.standard_normal((6, 5)), rng.standard_normal((4, 6))]
    b = [np.zeros(6), np.zeros(4)]
    x = rng.standard_normal((3, 5))
    a1, _ = H.mlp_forward(x, W, b)
    a2, _ = H.mlp_forward(3.5 * x, W, b)
    np.testing.assert_allclose(a2[-1], 3.5 * a1[-1], rtol=1e-13)


@pytest.mark.parametrize("gated", [False, True])
def test_mlp_backward_matches_autograd(gated):
    rng = np.random.default_rng(4)
    p = _params(rng, [9, 7], gated, 3, 6)
    x = rng.standard_normal((5, 6))
    ga = rng.standard_normal((5, 7))
    a, _ = H.mlp_forward(x, p["W"], p["b"], p.get("G"), p.get("c"))
    gx, gW, gb, gG, gc = H.mlp_backward(a, p["W"], p["b"], p.get("G"), p.get("c"), ga)
    tx = torch.from_numpy(x).requires_grad_()
    tW = [torch.from_numpy(w).requires_grad_() for w in p["W"]]
    tb = [torch.from_numpy(v).requires_grad_() for v in p["b"]]
    tG = [torch.from_numpy(g).requires_grad_() for g in p["G"]] if gated else None
    tc = [torch.tensor(float(v), dtype=torch.float64, requires_grad=True) for v in p["c"]] if gated else None
    t = tx
    for l in range(2):
        out = torch.relu(t @ tW[l].T + tb[l])
        if gated:
            out = out * torch.sigmoid(t @ tG[l] + tc[l])[:, None]
        t = out
    (t * torch.from_numpy(ga)).sum().backward()
    np.testing.assert_allclose(gx, tx.grad.numpy(), rtol=1e-12, atol=1e-13)
    for l in range(2):
        np.testing.assert_allclose(gW[l], tW[l].grad.numpy(), rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(gb[l], tb[l].grad.numpy(), rtol=1e-12, atol=1e-13)
        if gated:
            np.testing.assert_allclose(gG[l], tG[l].grad.numpy(), rtol=1e-12, atol=1e-13)
            assert gc[l] == pytest.approx(tc[l].grad.item(), rel=1e-12, abs=1e-13)


# ---------------------------------------------------------------------------
# Isotonic calibration
# ---------------------------------------------------------------------------

def test_bucket_worked_example():
    """K = 4, lo = -1, step = 0.5, y = 0.2: t = 1.2 lies in bucket 2 (1.2 - 1.0 > 0,
    1.2 - 1.5 < 0), so v = (0.5, 0.5, 0.2, 0)."""
    v, k = H.bucket_lengths(np.array([0.2]), -1.0, 0.5, 4)
    assert k[0] == 2
    np.testing.assert_allclose(v[0], [0.5, 0.5, 0.2, 0.0], atol=1e-15)
    y = H.calibrate(np.array([0.2]), np.zeros((1, 4)), np.array([1.0, 2.0, 3.0, 4.0]), 0.25, -1.0, 0.5)
    assert y[0] == pytest.approx(0.25 + 0.5 + 1.0 + 0.6)


@pytest.mark.parametrize("K,lo,step", [(37, -3.0, 0.17), (16, -3.0, 0.25)])
def test_bucket_index_is_searchsorted_in_float32(K, lo, step):
    """(The second case hits every bound exactly: a logit on a bound belongs to the
    bucket below it.)"""
    rng = np.random.default_rng(5)
    y = np.concatenate([rng.uniform(-6, 6, 2000), lo + step * np.arange(K + 2)])
    k = H.bucket_index(y, lo, step, K)
    t32 = y.astype(np.float32) - np.float32(lo)
    bounds = (np.float32(step) * np.arange(1, K, dtype=np.float32)).astype(np.float32)
    np.testing.assert_array_equal(k, np.searchsorted(bounds, t32, side="left"))
    assert k.min() == 0 and k.max() == K - 1


def test_unit_slopes_give_the_shifted_logit():
    """ReLU(e_i + w_i) = 1 everywhere: y_cal = b + (y - lo) on the whole line, the
    first and last buckets extending the line below lo and above lo + K*step."""
    y = np.linspace(-5, 5, 401)
    K = 6
    out = H.calibrate(y, np.zeros((y.size, K)), np.ones(K), 0.7, -1.0, 0.4)
    np.testing.assert_allclose(out, 0.7 + (y + 1.0), rtol=1e-13, atol=1e-13)


def test_calibration_is_isotonic_and_continuous():
    rng = np.random.default_rng(6)
    K, lo, step = 9, -1.5, 0.35
    e = np.repeat(rng.standard_normal((1, K)), 4001, axis=0)
    w = rng.standard_normal(K)
    y = np.linspace(-4, 4, 4001)
    out = H.calibrate(y, e, w, 0.1, lo, step)
    assert np.all(np.diff(out) >= -1e-12), "calibrated logit must not decrease"
    # continuity at every bucket bound: left and right limits agree
    # (1e-6 is a few float32 spacings here, so the two sides take different buckets)
    for j in range(1, K):
        yb = lo + step * j
        left = H.calibrate(np.array([yb - 1e-6]), e[:1], w, 0.1, lo, step)
        right = H.calibrate(np.array([yb + 1e-6]), e[:1], w, 0.1, lo, step)
        assert H.bucket_index(np.array([yb - 1e-6]), lo, step, K)[0] == j - 1
        assert H.bucket_index(np.array([yb + 1e-6]), lo, step, K)[0] == j
        assert abs(left[0] - right[0]) < 1e-5


def test_calibration_is_the_integral_of_the_bucket_slopes():
    """For y >= lo: y_cal - b = integral from lo to y of ReLU(e_i(u) + w_i(u)) du,
    i(u) = the bucket holding u (floor((u - lo)/step), clipped to K-1), by a fine
    midpoint sum."""
    rng = np.random.default_rng(7)
    K, lo, step = 7, -1.0, 0.3
    e = rng.standard_normal(K)
    w = rng.standard_normal(K)
    slope = np.maximum(e + w, 0.0)
    for y in [-1.0 + 1e-3, -0.65, 0.1, 0.77, 1.1, 2.5]:
        n = 200000
        h = (y - lo) / n
        u = lo + h * (np.arange(n) + 0.5)
        idx = np.minimum(np.floor((u - lo) / step).astype(np.int64), K - 1)
        integral = np.sum(slope[idx]) * h
        got = H.calibrate(np.array([y]), e[None, :], w, 0.4, lo, step)[0] - 0.4
        assert got == pytest.approx(integral, abs=2 * step * slope.max() / n * K + 1e-9)


def test_calibration_backward_finite_differences():
    rng = np.random.default_rng(8)
    K, lo, step, B = 6, -1.0, 0.5, 40
    y = rng.uniform(-2.5, 3.0, B)
    # keep every logit away from a bucket bound so the difference quotient sees one piece
    frac = (y - lo) / step - np.floor((y - lo) / step)
    y = np.where(np.minimum(frac, 1 - frac) < 0.05, y + 0.2 * step, y)
    e = rng.standard_normal((B, K))
    w = rng.standard_normal(K)
    g = rng.standard_normal(B)
    gy, ge, gw, gb = H.calibrate_backward(y, e, w, lo, step, g)
    f = lambda yy, ee, ww, bb: np.sum(g * H.calibrate(yy, ee, ww, bb, lo, step))
    hstep = 1e-6
    num_y = np.array([(f(y + hstep * (np.arange(B) == i), e, w, 0.0) - f(y - hstep * (np.arange(B) == i), e, w, 0.0))
                      / (2 * hstep) for i in range(B)])
    np.testing.assert_allclose(gy, num_y, rtol=1e-6, atol=1e-8)
    for i in range(K):
        dw = np.zeros(K)
        dw[i] = hstep
        if np.any(np.abs(e[:, i] + w[i]) < 1e-4):
            continue
        assert gw[i] == pytest.approx((f(y, e, w + dw, 0.0) - f(y, e, w - dw, 0.0)) / (2 * hstep), rel=1e-6, abs=1e-8)
    for bi in range(0, B, 7):
        for i in range(K):
            de = np.zeros_like(e)
            de[bi, i] = hstep
            if abs(e[bi, i] + w[i]) < 1e-4:
                continue
            num = (f(y, e + de, w, 0.0) - f(y, e - de, w, 0.0)) / (2 * hstep)
            assert ge[bi, i] == pytest.approx(num, rel=1e-6, abs=1e-8)
    assert gb == pytest.approx(g.sum(), rel=1e-14)


# ---------------------------------------------------------------------------
# Log loss and the whole head
# ---------------------------------------------------------------------------

def test_logloss_matches_torch_bce():
    rng = np.random.default_rng(9)
    z = np.concatenate([rng.standard_normal(50) * 4, [-60.0, 60.0, 0.0]])
    lab = rng.integers(0, 2, z.size).astype(np.float64)
    loss, grad = H.logloss(z, lab)
    tz = torch.from_numpy(z).requires_grad_()
    tl = torch.nn.functional.binary_cross_entropy_with_logits(tz, torch.from_numpy(lab), reduction="none")
    np.testing.assert_allclose(loss, tl.detach().numpy(), rtol=1e-13, atol=1e-15)
    tl.sum().backward()
    np.testing.assert_allclose(grad, tz.grad.numpy(), rtol=1e-13, atol=1e-15)
    assert H.logloss(np.array([0.0]), np.array([1.0]))[0][0] == pytest.approx(np.log(2.0))


@pytest.mark.parametrize("gated", [False, True])
def test_head_backward_finite_differences(gated):
    rng = np.random.default_rng(10 + gated)
    K, B = 5, 6
    p = _params(rng, [7, 5], gated, K, 4)
    p["e"] = 0.3 * rng.standard_normal((B, K))
    x = rng.standard_normal((B, 4))
    g = rng.standard_normal(B)
    out = H.head_backward(x, p, g)
    # keep logits off bucket bounds and pre-activations off zero for the difference quotients
    fwd = H.head_forward(x, p)
    t = (fwd["y"] - p["lo"]) / p["step"]
    assert np.min(np.abs(t - np.round(t))) > 1e-3

    def f(**kw):
        q = dict(p)
        q.update(kw)
        return np.sum(g * H.head_forward(kw.get("x", x), q)["y_cal"])

    h = 1e-6
    for i in range(B):
        for j in range(4):
            dx = np.zeros_like(x)
            dx[i, j] = h
            num = (f(x=x + dx) - f(x=x - dx)) / (2 * h)
            assert out["x"][i, j] == pytest.approx(num, rel=1e-5, abs=1e-7)
    for l in range(2):
        for (i, j) in [(0, 0), (1, 2), (3, 1)]:
            Wp = [w.copy() for w in p["W"]]
            Wm = [w.copy() for w in p["W"]]
            Wp[l][i, j] += h
            Wm[l][i, j] -= h
            num = (f(W=Wp) - f(W=Wm)) / (2 * h)
            assert out["W"][l][i, j] == pytest.approx(num, rel=1e-5, abs=1e-7)
        bp = [v.copy() for v in p["b"]]
        bm = [v.copy() for v in p["b"]]
        bp[l][1] += h
        bm[l][1] -= h
        assert out["b"][l][1] == pytest.approx((f(b=bp) - f(b=bm)) / (2 * h), rel=1e-5, abs=1e-7)
        if gated:
            Gp = [v.copy() for v in p["G"]]
            Gm = [v.copy() for v in p["G"]]
            Gp[l][2] += h
            Gm[l][2] -= h
            assert out["G"][l][2] == pytest.approx((f(G=Gp) - f(G=Gm)) / (2 * h), rel=1e-5, abs=1e-7)
            cp = list(p["c"])
            cm = list(p["c"])
            cp[l] += h
            cm[l] -= h
            assert out["c"][l] == pytest.approx((f(c=cp) - f(c=cm)) / (2 * h), rel=1e-5, abs=1e-7)
    wo = p["w_out"]
    for j in range(5):
        d = np.zeros_like(wo)
        d[j] = h
        assert out["w_out"][j] == pytest.approx((f(w_out=wo + d) - f(w_out=wo - d)) / (2 * h), rel=1e-5, abs=1e-7)
    assert out["b_out"] == pytest.approx((f(b_out=p["b_out"] + h) - f(b_out=p["b_out"] - h)) / (2 * h), rel=1e-5)
    assert out["cal_b"] == pytest.approx(g.sum(), rel=1e-14)


def test_rounded_activations_only_change_the_stored_values():
    """round_act is applied to the stored activations only: with an identity rounding
    the results are unchanged, and with bf16 rounding every a_l is a bf16 value and the
    backward's masks follow the rounded activations (z recomputed from them)."""
    import oracle
    rng = np.random.default_rng(12)
    p = _params(rng, [16, 8], True, 4, 8)
    x = rng.standard_normal((5, 8))
    a0, _ = H.mlp_forward(x, p["W"], p["b"], p["G"], p["c"])
    a1, _ = H.mlp_forward(x, p["W"], p["b"], p["G"], p["c"], round_act=lambda v: v)
    for u, v in zip(a0, a1):
        np.testing.assert_array_equal(u, v)
    ar, _ = H.mlp_forward(x, p["W"], p["b"], p["G"], p["c"], round_act=oracle.round_bf16)
    for l in (1, 2):
        np.testing.assert_array_equal(ar[l], oracle.round_bf16(ar[l]).astype(np.float64))
        assert np.max(np.abs(ar[l] - a0[l])) <= 2.0 ** -8 * np.max(np.abs(a0[l])) * 2
