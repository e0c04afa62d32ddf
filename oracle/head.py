"""CPU oracle for the layers after the cross stack -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this module; the product library and its Python binding never do.

Float64 numpy; numpy's matrix product is the only library step. It follows:
  - section "Dense Gating and Large MLP": a stack of wide ReLU layers after the
    interaction layers, each hidden layer gated (the gate idea of GateNet,
    applied to hidden layers at negligible extra matrix cost);
  - section "Isotonic Calibration Layer", equation (calibration): the logit is
    cut into buckets of width `step`, each bucket i carries a trainable weight
    w_i plus a per-sample embedding value e_i, and the calibrated logit is
    b + sum_i ReLU(e_i + w_i) * v_i, with v_i = step for every bucket below the
    logit's bucket k, v_k = the remainder of the logit inside bucket k;
  - a log loss on the calibrated logit (the paper's tasks are binary).

Readings where the paper is silent (each is a choice of this library):
  - gate: hidden layer l computes a_l = ReLU(W_l a_{l-1} + b_l) * sigmoid(g_l . a_{l-1} + c_l),
    one scalar gate per sample and layer from the layer's own input (the
    vector-wise gate: one extra row of matrix work per layer);
  - the logit is y = w_o . a_L + b_o;
  - buckets start at `lo`: t = y - lo, and k is the largest j in [0, K-1]
    with t - step*j > 0, or 0 when there is none; so below lo the first bucket
    and above lo + K*step the last bucket extend linearly (v_0 = t <= 0 there,
    v_{K-1} = t - step*(K-1) > step). The decision k is taken in float32
    (t and the bucket bounds step*j rounded to float32), as the device does;
    the values are float64;
  - ReLU'(0) = 0;
  - e is an input [B, K] (the calibration-feature embedding made upstream);
    its gradient is returned;
  - loss_b = softplus(y_cal) - label * y_cal, its gradient sigmoid(y_cal) - label.

ReLU masks and the bucket index are decisions taken by floating point. To take
them on the same values as a device that keeps its hidden activations in a
narrower storage type, `round_act` (optional) is applied to every stored hidden
activation a_1 .. a_L; everything else stays float64.
"""
from __future__ import annotations

from typing import Callable, List, Optional, Sequence

import numpy as np


def sigmoid(z):
    z = np.asarray(z, dtype=np.float64)
    out = np.empty_like(z)
    pos = z >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-z[pos]))
    ez = np.exp(z[~pos])
    out[~pos] = ez / (1.0 + ez)
    return out


def softplus(z):
    z = np.asarray(z, dtype=np.float64)
    return np.maximum(z, 0.0) + np.log1p(np.exp(-np.abs(z)))


# ---------------------------------------------------------------------------
# Gated MLP
# ---------------------------------------------------------------------------

def mlp_forward(x, W: Sequence, b: Sequence, G: Optional[Sequence] = None, c: Optional[Sequence] = None,
                round_act: Optional[Callable] = None):
    """a_0 = x; a_l = ReLU(a_{l-1} W_l^T + b_l) [* sigmoid(a_{l-1} g_l + c_l)].

    x [B, n_0]; W[l] [n_l, n_{l-1}]; b[l] [n_l]; G[l] [n_{l-1}]; c[l] scalar;
    round_act(a) -> a, applied to each a_l (l >= 1) before it is used or returned.
    Returns (a, s): activations a_0 .. a_L and gate logits s_1 .. s_L (empty when ungated).
    """
    a = [np.asarray(x, dtype=np.float64)]
    s = []
    for l in range(len(W)):
        prev = a[-1]
        z = prev @ np.asarray(W[l], dtype=np.float64).T + np.asarray(b[l], dtype=np.float64)
        act = np.maximum(z, 0.0)
        if G is not None:
            sl = prev @ np.asarray(G[l], dtype=np.float64) + float(c[l])
            act = act * sigmoid(sl)[:, None]
            s.append(sl)
        if round_act is not None:
            act = np.asarray(round_act(act), dtype=np.float64)
        a.append(act)
    return a, s


def mlp_backward(a: List, W: Sequence, b: Sequence, G: Optional[Sequence], c: Optional[Sequence], ga_top):
    """Chain rule through mlp_forward, given dLoss/da_L.

    Returns (g_x, gW, gb, gG, gc); gG and gc are None when ungated.
    """
    L = len(W)
    ga = np.asarray(ga_top, dtype=np.float64)
    gW, gb = [None] * L, [None] * L
    gG = [None] * L if G is not None else None
    gc = [None] * L if G is not None else None
    for l in range(L - 1, -1, -1):
        prev = a[l]
        Wl = np.asarray(W[l], dtype=np.float64)
        z = prev @ Wl.T + np.asarray(b[l], dtype=np.float64)
        relu = np.maximum(z, 0.0)
        if G is not None:
            Gl = np.asarray(G[l], dtype=np.float64)
            rho = sigmoid(prev @ Gl + float(c[l]))
            g_relu = ga * rho[:, None]
            g_rho = np.sum(ga * relu, axis=1)
            g_s = g_rho * rho * (1.0 - rho)
        else:
            g_relu = ga
        g_z = g_relu * (z > 0.0)
        gW[l] = g_z.T @ prev
        gb[l] = g_z.sum(axis=0)
        ga = g_z @ Wl
        if G is not None:
            gG[l] = g_s @ prev
            gc[l] = g_s.sum()
            ga = ga + np.outer(g_s, Gl)
    return ga, gW, gb, gG, gc


# ---------------------------------------------------------------------------
# Isotonic calibration
# ---------------------------------------------------------------------------

def bucket_index(y, lo: float, step: float, K: int):
    """Bucket k of each logit: the largest j in [0, K-1] with t - step*j > 0 (t = y - lo),
    or 0 when there is none. Decided in float32: t = fl32(fl32(y) - fl32(lo)) against the
    float32 bounds fl32(fl32(step) * j)."""
    t32 = (np.asarray(y, dtype=np.float64).astype(np.float32) - np.float32(lo)).astype(np.float32)
    k = np.zeros(t32.shape, dtype=np.int64)
    for j in range(1, K):
        bound = np.float32(np.float32(step) * np.float32(j))
        k += (t32 > bound).astype(np.int64)
    return k


def bucket_lengths(y, lo: float, step: float, K: int):
    """v [B, K]: step for buckets below k, the remainder t - step*k for bucket k, 0 above."""
    y = np.asarray(y, dtype=np.float64)
    k = bucket_index(y, lo, step, K)
    t = y - lo
    v = np.zeros(y.shape + (K,), dtype=np.float64)
    for i in range(K):
        below = i < k
        v[below, i] = step
        here = i == k
        v[here, i] = t[here] - step * k[here]
    return v, k


def calibrate(y, e, w, bc: float, lo: float, step: float):
    """y_cal = bc + sum_i ReLU(e_i + w_i) * v_i  (y [B], e [B, K], w [K])."""
    e = np.asarray(e, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    K = w.shape[0]
    v, _ = bucket_lengths(y, lo, step, K)
    return float(bc) + np.sum(np.maximum(e + w, 0.0) * v, axis=1)


def calibrate_backward(y, e, w, lo: float, step: float, g_cal):
    """Gradients of calibrate() given dLoss/dy_cal: (g_y, g_e, g_w, g_bc)."""
    e = np.asarray(e, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    g_cal = np.asarray(g_cal, dtype=np.float64)
    K = w.shape[0]
    v, k = bucket_lengths(y, lo, step, K)
    pre = e + w
    g_e = g_cal[:, None] * (pre > 0.0) * v
    g_w = g_e.sum(axis=0)
    g_bc = g_cal.sum()
    rows = np.arange(pre.shape[0])
    g_y = g_cal * np.maximum(pre[rows, k], 0.0)
    return g_y, g_e, g_w, g_bc


def logloss(y_cal, label):
    """Per-sample log loss on the calibrated logit and its gradient."""
    y_cal = np.asarray(y_cal, dtype=np.float64)
    label = np.asarray(label, dtype=np.float64)
    return softplus(y_cal) - label * y_cal, sigmoid(y_cal) - label


# ---------------------------------------------------------------------------
# The whole head
# ---------------------------------------------------------------------------

def head_forward(x, p: dict, round_act: Optional[Callable] = None):
    """p: W, b, (G, c when gated), w_out, b_out, cal_w, cal_b, lo, step; plus e [B, K].
    Returns dict(a, s, y, y_cal)."""
    a, s = mlp_forward(x, p["W"], p["b"], p.get("G"), p.get("c"), round_act)
    y = a[-1] @ np.asarray(p["w_out"], dtype=np.float64) + float(p["b_out"])
    y_cal = calibrate(y, p["e"], p["cal_w"], p["cal_b"], p["lo"], p["step"])
    return {"a": a, "s": s, "y": y, "y_cal": y_cal}


def head_backward(x, p: dict, g_cal, round_act: Optional[Callable] = None):
    """Gradients of every input and parameter of head_forward given dLoss/dy_cal
    (with round_act, the gradients at the rounded activations)."""
    f = head_forward(x, p, round_act)
    g_y, g_e, g_w, g_bc = calibrate_backward(f["y"], p["e"], p["cal_w"], p["lo"], p["step"], g_cal)
    aL = f["a"][-1]
    w_out = np.asarray(p["w_out"], dtype=np.float64)
    g_wout = g_y @ aL
    g_bout = g_y.sum()
    ga = np.outer(g_y, w_out)
    g_x, gW, gb, gG, gc = mlp_backward(f["a"], p["W"], p["b"], p.get("G"), p.get("c"), ga)
    return {"x": g_x, "W": gW, "b": gb, "G": gG, "c": gc, "w_out": g_wout, "b_out": g_bout,
            "e": g_e, "cal_w": g_w, "cal_b": g_bc, "y": f["y"], "y_cal": f["y_cal"]}
