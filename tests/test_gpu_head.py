"""GPU head (gated MLP, logit, isotonic calibration, log loss) vs the float64 oracle.

Two oracles. The plain one is the definition in float64 throughout (the same bf16
parameters and inputs, no rounding of anything it computes); the device must match
it within the bars of the bf16 cross stack (2e-2 forward, 5e-2 gradients). The
emulating one rounds its hidden activations to f16 (oracle.round_f16), the copy the
device's forward reads, so that ReLU masks and the calibration bucket are decided
on the values the device uses (all its arithmetic is float64); against it the bars
are tighter (2e-3 forward, 1e-2 gradients: the device keeps the pre-activation
gradients G in bf16, and its weight-gradient products read bf16 activations).

Small shapes are compared in full; the Feed-sized head (4 x 3500, stored as
4 x 3504 with zero padding) runs at the full batch in the launch configuration
the benchmark uses and is compared on sampled rows (the upstream gradient is
zero elsewhere, so every parameter gradient is that of the sampled rows).
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import head as OH
from gpu_helpers import need_gpu, relerr, sample_rows, to_np
from paper_2402_06859_amd.rdcn import RDCN_ERR_ARG, Rdcn, RdcnError, config_for, make_head_config
from paper_2402_06859_amd.step import DeviceHead
from paper_2402_06859_amd.synth import HEADS, WORKLOADS, HeadSpec, Workload, make_head_inputs

pytestmark = pytest.mark.gpu

Y_TOL = 2e-3      # logits / calibrated logits (f16 rounding of activations on both sides)
GRAD_TOL = 1e-2   # parameter and input gradients (device G in bf16)
CAL_TOL = 1e-5    # the calibration bias gradient (a float sum of the upstream gradient)
PLAIN_Y_TOL, PLAIN_GRAD_TOL = 2e-2, 5e-2  # against the plain float64 definition


def oracle_params(hinp: dict, head: HeadSpec) -> dict:
    f = lambda t: t.float().numpy().astype(np.float64)
    p = {"W": [f(w) for w in hinp["W"]], "b": [f(v) for v in hinp["b"]], "w_out": f(hinp["w_out"]),
         "b_out": float(hinp["b_out"].float()[0]), "cal_w": f(hinp["cal_w"]), "cal_b": float(hinp["cal_b"][0]),
         "lo": head.lo, "step": head.step, "e": f(hinp["e"])}
    if head.gated:
        p["G"] = [f(g) for g in hinp["G"]]
        p["c"] = [float(c.float()[0]) for c in hinp["c"]]
    return p


def run_head(wl: Workload, head: HeadSpec, B: int, rows=None, seed=None, hinp=None, round_act=oracle.round_f16):
    """Device forward + backward with upstream g_cal (zero outside `rows`), oracle on `rows`
    (round_act=None: the plain float64 definition)."""
    print("head", head.name, head.hidden, "gated", head.gated, "K", head.buckets, "B", B, "d", wl.d, flush=True)
    hinp = make_head_inputs(wl, head, batch=B, seed=seed) if hinp is None else hinp
    rows = np.arange(B) if rows is None else rows
    g = torch.zeros(B, dtype=torch.float32)
    g[torch.from_numpy(rows)] = hinp["g_cal"][torch.from_numpy(rows)]
    hinp = dict(hinp, g_cal=g)
    lib = Rdcn(config_for(wl, max(B, 1)))
    dh = DeviceHead(lib, head, hinp, B)
    dh.forward()
    dh.backward(g_cal=dh.g_cal_in)
    torch.cuda.synchronize()
    p = oracle_params(hinp, head)
    x = hinp["x"].float().numpy().astype(np.float64)
    p_rows = dict(p, e=p["e"][rows])
    g64 = g.numpy().astype(np.float64)
    ref = OH.head_backward(x[rows], p_rows, g64[rows], round_act=round_act)
    ref["scale"] = sum_scale(x, p, g64, rows, round_act)
    return dh, ref, rows, p


def sum_scale(x, p, g, rows, round_act=oracle.round_f16) -> dict:
    """Sum over rows of |per-row contribution| of each scalar gradient (gate biases, b_out):
    the scale of the summation error bound. A scalar gradient can be a nearly cancelling
    sum (0.01 out of terms whose magnitudes add up to 14 on the ragged case), so it is
    compared against this scale rather than against its own size."""
    acc = None
    for r in rows:
        o = OH.head_backward(x[r:r + 1], dict(p, e=p["e"][r:r + 1]), g[r:r + 1], round_act=round_act)
        v = {"b_out": abs(o["b_out"])}
        if o["c"] is not None:
            for l, c in enumerate(o["c"]):
                v["c%d" % l] = abs(c)
        acc = v if acc is None else {k: acc[k] + v[k] for k in acc}
    return acc


def compare(dh: DeviceHead, ref: dict, rows, gated: bool, grad_tol=GRAD_TOL, y_tol=Y_TOL):
    scale = ref["scale"]
    errs = {"y": relerr(to_np(dh.y)[rows], ref["y"]), "y_cal": relerr(to_np(dh.y_cal)[rows], ref["y_cal"])}
    assert errs["y"] <= y_tol and errs["y_cal"] <= y_tol, errs
    gerr = {"x": relerr(to_np(dh.grad_x)[rows], ref["x"]), "e": relerr(to_np(dh.grad_e)[rows], ref["e"]),
            "w_out": relerr(to_np(dh.grads["w_out"]), ref["w_out"]),
            "b_out": abs(float(to_np(dh.grads["b_out"])[0]) - ref["b_out"]) / scale["b_out"],
            "cal_w": relerr(to_np(dh.grads["cal_w"]), ref["cal_w"]),
            "cal_b": relerr(to_np(dh.grads["cal_b"]), [ref["cal_b"]])}
    for l in range(len(ref["W"])):
        gerr["W%d" % l] = relerr(to_np(dh.grads["W"][l]), ref["W"][l])
        gerr["b%d" % l] = relerr(to_np(dh.grads["b"][l]), ref["b"][l])
        if gated:
            gerr["G%d" % l] = relerr(to_np(dh.grads["G"][l]), ref["G"][l])
            gerr["c%d" % l] = abs(float(to_np(dh.grads["c"][l])[0]) - ref["c"][l]) / scale["c%d" % l]
    print("y %.3g  y_cal %.3g  max grad %.3g (%s)" % (errs["y"], errs["y_cal"], max(gerr.values()),
                                                      max(gerr, key=gerr.get)), flush=True)
    # cal_b sums g_cal alone; grad_e and cal_w carry v_k = t - step*k and so the logit's error
    assert gerr["cal_b"] <= CAL_TOL and gerr["e"] <= y_tol and gerr["cal_w"] <= y_tol, gerr
    bad = {k: v for k, v in gerr.items() if not v <= grad_tol}
    assert not bad, "gradient rel err above %.3g: %s" % (grad_tol, bad)
    if len(rows) < dh.B:
        others = np.setdiff1d(np.arange(dh.B), rows)
        assert not np.any(to_np(dh.grad_x)[others]) and not np.any(to_np(dh.grad_e)[others])


# d = 5 * 24 + 40 = 160: not a tile multiple
RAGGED = Workload("ragged", 11, 300, 5, 50_000, 250, 24, 40, 2, 40, True, "bf16", "sum", 1.1)


@pytest.mark.parametrize("gated", [True, False])
def test_ragged_small_head(gated):
    """batch 300, widths 40 and 24 (no tile multiples), 9 buckets over a narrow range so
    that many logits fall below lo or above lo + K*step."""
    need_gpu()
    head = HeadSpec("ragged", (40, 24), gated=gated, buckets=9, lo=-0.5, step=0.1)
    dh, ref, rows, _ = run_head(RAGGED, head, 300)
    compare(dh, ref, rows, gated)
    k = OH.bucket_index(ref["y"], head.lo, head.step, head.buckets)
    assert np.any(k == 0) and np.any(k == head.buckets - 1) and np.any((k > 0) & (k < head.buckets - 1))


@pytest.mark.parametrize("K", [1, 64, 200])
def test_bucket_counts(K):
    """One bucket (pure linear map of t), exactly one wave of bounds, several rounds of lanes."""
    need_gpu()
    head = HeadSpec("buckets", (64, 32), gated=True, buckets=K, lo=-3.0, step=6.0 / K)
    dh, ref, rows, _ = run_head(RAGGED, head, 130)
    compare(dh, ref, rows, True)


def test_small_head_on_small_workload_width():
    """d = 1856 input (the small cross stack's width), widths 256 and 128, full batch."""
    need_gpu()
    wl = WORKLOADS["small"]
    dh, ref, rows, _ = run_head(wl, HEADS["small"], wl.batch, rows=sample_rows(wl.batch, 64))
    compare(dh, ref, rows, True)


def test_large_mlp_full_batch_sampled():
    """Feed's Large MLP (4 x 3500, gated) on the small workload's batch of 4096."""
    need_gpu()
    wl = WORKLOADS["small"]
    dh, ref, rows, _ = run_head(wl, HEADS["lmlp"], wl.batch, rows=sample_rows(wl.batch, 24))
    compare(dh, ref, rows, True)
    # the padding units stay inert: zero activations never reach a gradient
    for l, n in enumerate(HEADS["lmlp"].hidden):
        gW = to_np(dh.grads["W"][l])
        assert not np.any(gW[n:]) and not np.any(to_np(dh.grads["b"][l])[n:])


@pytest.mark.parametrize("case", ["ragged_gated", "ragged_plain", "lmlp"])
def test_head_against_plain_float64_definition(case):
    """The device against the head computed in float64 from the same bf16 parameters and
    inputs with nothing rounded, at the bf16 bars (2e-2 forward, 5e-2 gradients): the
    ragged head, gated and plain (many logits outside the bucket range), and Feed's
    Large MLP (4 x 3500, gated) on 64 sampled rows of a 4096 batch. On the latter,
    activations rounded to bf16 would flip enough ReLU masks in the deeper layers to
    move the gradients by about 6% from the definition; with the f16 copies the
    float64 emulation of the device's rounding is 2.2% away (x and W0 gradients)."""
    need_gpu()
    if case == "lmlp":
        wl, head, B = WORKLOADS["small"], HEADS["lmlp"], WORKLOADS["small"].batch
        rows = sample_rows(B, 64)
    else:
        wl, B, rows = RAGGED, 300, None
        head = HeadSpec("ragged", (40, 24), gated=case == "ragged_gated", buckets=9, lo=-0.5, step=0.1)
    dh, ref, rows, _ = run_head(wl, head, B, rows=rows, round_act=None)
    compare(dh, ref, rows, head.gated, grad_tol=PLAIN_GRAD_TOL, y_tol=PLAIN_Y_TOL)


def test_logloss_matches_oracle():
    need_gpu()
    rng = np.random.default_rng(3)
    z = np.concatenate([rng.standard_normal(1000).astype(np.float32) * 5, np.float32([-90, 90, 0, -1e-3])])
    lab = rng.integers(0, 2, z.size).astype(np.float32)
    lib = Rdcn(config_for(RAGGED, z.size))
    zt, lt = torch.from_numpy(z).cuda(), torch.from_numpy(lab).cuda()
    loss = torch.empty_like(zt)
    grad = torch.empty_like(zt)
    lib.head_logloss(z.size, zt, lt, 0.5, loss, grad)
    torch.cuda.synchronize()
    ref_loss, ref_grad = OH.logloss(z.astype(np.float64), lab.astype(np.float64))
    np.testing.assert_allclose(to_np(loss), ref_loss, rtol=2e-6, atol=1e-6)
    np.testing.assert_allclose(to_np(grad), 0.5 * ref_grad, rtol=2e-6, atol=1e-7)


def test_batch_zero_and_one():
    need_gpu()
    head = HeadSpec("tiny", (16, 8), gated=True, buckets=5, lo=-1.0, step=0.5)
    dh, ref, rows, _ = run_head(RAGGED, head, 1)
    compare(dh, ref, rows, True)
    hinp = make_head_inputs(RAGGED, head, batch=4)
    lib = Rdcn(config_for(RAGGED, 4))
    dh = DeviceHead(lib, head, hinp, 4)
    for t in list(dh.grads.values()):
        for u in (t if isinstance(t, list) else [t]):
            u.fill_(7.0)
    dh.B = 0
    dh.forward()
    dh.backward(g_cal=dh.g_cal_in)
    torch.cuda.synchronize()
    for t in list(dh.grads.values()):
        for u in (t if isinstance(t, list) else [t]):
            assert not torch.any(u), "an empty batch has zero gradients"


def test_deterministic_rerun():
    need_gpu()
    wl = WORKLOADS["small"].with_(batch=512)
    head = HEADS["small"]
    hinp = make_head_inputs(wl, head)
    outs = []
    for _ in range(2):
        lib = Rdcn(config_for(wl))
        dh = DeviceHead(lib, head, hinp, wl.batch)
        dh.forward()
        dh.logloss()
        dh.backward()
        torch.cuda.synchronize()
        outs.append([dh.y_cal.cpu(), dh.grad_x.cpu().view(torch.int16), dh.grad_e.cpu()] +
                    [t.cpu() for k in ("W", "b", "G", "c") for t in dh.grads[k]] +
                    [dh.grads[k].cpu() for k in ("w_out", "b_out", "cal_w", "cal_b")])
    for a, b in zip(*outs):
        assert torch.equal(a, b)


def test_head_needs_a_bf16_model():
    need_gpu()
    from paper_2402_06859_amd.rdcn import RDCN_ERR_UNSUPPORTED
    lib = Rdcn(config_for(WORKLOADS["tiny"], 8))  # float storage
    with pytest.raises(RdcnError) as ei:
        lib.head_configure(make_head_config([16], True, 4, 0.0, 1.0))
    assert ei.value.status == RDCN_ERR_UNSUPPORTED


def test_head_argument_errors():
    need_gpu()
    lib = Rdcn(config_for(RAGGED, 8))
    for bad in [make_head_config([], True, 4, 0.0, 1.0), make_head_config([12], True, 4, 0.0, 1.0),
                make_head_config([16], True, 0, 0.0, 1.0), make_head_config([16], True, 4, 0.0, 0.0),
                make_head_config([16], 2, 4, 0.0, 1.0)]:
        with pytest.raises(RdcnError) as ei:
            lib.head_configure(bad)
        assert ei.value.status == RDCN_ERR_ARG


def test_head_f16_overflow_is_reported():
    """The head's hidden activations go to the next layer as f16: an input of 1e6 (exact
    enough in bf16) drives a_1 beyond the f16 range, and the forward reports
    RDCN_ERR_RANGE through the device error word."""
    need_gpu()
    from paper_2402_06859_amd.rdcn import RDCN_ERR_RANGE, RDCN_OK
    head = HeadSpec("ovf", (16, 8), gated=False, buckets=4, lo=-1.0, step=0.5)
    hinp = make_head_inputs(RAGGED, head, batch=32)
    lib = Rdcn(config_for(RAGGED, 32))
    dh = DeviceHead(lib, head, dict(hinp, x=torch.full_like(hinp["x"], 1.0e6)), 32)
    dh.forward()
    torch.cuda.synchronize()
    assert lib.check_device_errors() == RDCN_ERR_RANGE
    dh2 = DeviceHead(lib, head, hinp, 32)
    dh2.forward()
    torch.cuda.synchronize()
    assert lib.check_device_errors() == RDCN_OK
