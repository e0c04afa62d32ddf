"""GPU Residual-DCN forward/backward (rdcn_forward / rdcn_backward) vs the fp64 oracle.

Small shapes are compared in full (ragged batch, ragged d, attention on/off,
several temperatures). Every workload is also run at its full batch in the
launch configuration the benchmark uses, and compared on sampled rows and on
whole 256-row tiles (the first, one in the middle, the last): the forward of a
row depends on that row only, and with an upstream gradient that is zero outside
the compared rows (dense on them) the weight gradients are exactly those of the
compared rows (other rows contribute exact zeros), which the oracle computes on
those rows alone (tests/oracle_pool.py splits them over worker processes).

Every tensor passes three gates (gpu_helpers.check_tensor): the normwise relative
error within the stated bar (2e-2 forward, 5e-2 gradients for bf16; 1e-5 / 1e-4
for float), every row and column, and every element, within a multiple of it on
the larger of their own and the tensor's typical scale (3x and 10x for the forward,
5x and 20x for gradients; the reasons are stated in gpu_helpers).
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import (FWD_TOL, GRAD_GATES, GRAD_TOL, check_tensor, need_gpu, oracle_x0, relerr, sample_rows,
                         tile_rows, to_np)
from oracle_pool import dcn_oracle
from paper_2402_06859_amd.step import DeviceBatch
from paper_2402_06859_amd.synth import WORKLOADS, Workload, make_inputs

pytestmark = pytest.mark.gpu


def host_weights(inp):
    return ([w.float().numpy() for w in inp["w_down"]], [w.float().numpy() for w in inp["u"]],
            [w.float().numpy() for w in inp["bias"]])


def run_full_compare(wl: Workload, seed=None, grad_rows=None, fwd_rows=None, bias_std=0.1, id_mode="scatter",
                     fwd_tol=None, grad_tol=None, pool=False):
    """Device gather + forward + backward at wl's batch; oracle forward on fwd_rows and
    backward on grad_rows (the upstream gradient is zero on the other rows). pool: run
    the oracle over worker processes (large row counts)."""
    inp = make_inputs(wl, seed=seed, bias_std=bias_std, id_mode=id_mode)
    B = inp["batch"]
    print("dcn", wl.name, "B", B, "d", wl.d, "r", wl.rank, "L", wl.num_layers, "attn", wl.attention,
          "act", wl.act_mode, "fwd rows", "all" if fwd_rows is None else len(fwd_rows),
          "grad rows", "all" if grad_rows is None else len(grad_rows), flush=True)
    if grad_rows is not None:  # upstream gradient only on the compared rows
        G = torch.zeros_like(inp["grad_out"])
        G[torch.from_numpy(grad_rows)] = inp["grad_out"][torch.from_numpy(grad_rows)]
        inp["grad_out"] = G
    db = DeviceBatch(wl, inp)
    db.gather()
    db.forward()
    db.backward()
    torch.cuda.synchronize()
    x0_ref = oracle_x0(wl, inp)
    W, U, b = host_weights(inp)
    rows = np.arange(B) if fwd_rows is None else fwd_rows
    grows = np.arange(B) if grad_rows is None else grad_rows
    G = inp["grad_out"].float().numpy()
    args = (wl.alpha, wl.beta, wl.temperature)
    if pool:
        same = np.array_equal(rows, grows)
        r = dcn_oracle(x0_ref[grows], W, U, b, G[grows], *args, parallel=wl.parallel)
        xL_g, (gx0, gW, gU, gb) = r[0], r[1:]
        xL = xL_g if same else dcn_oracle(x0_ref[rows], W, U, b, None, *args, parallel=wl.parallel, backward=False)
    else:
        xL = oracle.forward(x0_ref[rows], W, U, b, *args, parallel=wl.parallel)
        gx0, gW, gU, gb = oracle.backward(x0_ref[grows], W, U, b, G[grows], *args, parallel=wl.parallel)
    tol = FWD_TOL[wl.dtype] if fwd_tol is None else fwd_tol
    gtol = (1e-4 if wl.dtype == "f32" else GRAD_TOL) if grad_tol is None else grad_tol
    errs, bad = {}, []
    bad += check_tensor("x_L", to_np(db.x_out)[rows], xL, tol, errs)
    got_gx0 = to_np(db.grad_x0)
    bad += check_tensor("grad_x0", got_gx0[grows], gx0, gtol, errs, GRAD_GATES)
    if grad_rows is not None:
        others = np.setdiff1d(np.arange(B), grows)
        assert not np.any(got_gx0[others]), "rows without upstream gradient must get exact zeros"
    for l in range(wl.num_layers):
        bad += check_tensor("w_down%d" % l, to_np(db.g_w_down[l]), gW[l], gtol, errs, GRAD_GATES)
        bad += check_tensor("u%d" % l, to_np(db.g_u[l]), gU[l], gtol, errs, GRAD_GATES)
        bad += check_tensor("bias%d" % l, to_np(db.g_bias[l]), gb[l], gtol, errs, GRAD_GATES)
    worst = lambda key: max((e.get(key, 0.0), k) for k, e in errs.items() if k != "x_L")
    print("fwd norm %.3g row %.3g elem %.3g | grads: norm %.3g (%s) row %.3g col %.3g elem %.3g (%s)" % (
        errs["x_L"]["norm"], errs["x_L"]["row"], errs["x_L"]["elem"], *worst("norm"), worst("row")[0],
        worst("col")[0], *worst("elem")), flush=True)
    assert not bad, "; ".join(bad)
    return db


def test_tiny_full():
    need_gpu()
    run_full_compare(WORKLOADS["tiny"])


@pytest.mark.parametrize("attn,tau,beta", [(True, 1.0, 1.0), (True, 0.25, 1.0), (True, 4.0, 0.5), (False, 1.0, 1.0),
                                           (False, 1.0, 0.5)])
def test_ragged_small_shapes(attn, tau, beta):
    """batch 300 and d = 5*24 + 40 = 160 are not tile multiples; r = 40 is not a multiple of 16."""
    need_gpu()
    wl = Workload("ragged", 11, 300, 5, 50_000, 250, 24, 40, 2, 40, attn, "bf16", "sum", 1.1, temperature=tau)
    run_full_compare(wl.with_(skip_beta=beta))


@pytest.mark.parametrize("rank", [40, 256])
def test_attention_extreme_logits(rank):
    """tau = 1e-4 puts the exponent coefficients beyond f16 range, so the attention kernels
    compute the exponent arguments with FMAs instead of on the matrix cores (both the
    paired-tile form of waves with up to 8 tiles and the 16-tile form). One layer: its q
    and k come from bf16 inputs exactly, so the nearly one-hot softmax picks the same
    keys as the float64 oracle (with more layers, rounding the stored activations to
    bf16 moves near-ties)."""
    need_gpu()
    wl = Workload("extreme", 16, 200, 5, 50_000, 250, 24, 40, 1, rank, True, "bf16", "sum", 1.1, temperature=1e-4)
    run_full_compare(wl)


@pytest.mark.parametrize("mode,tol", [("hilo", 2e-3), ("f16", 5e-3)])
@pytest.mark.parametrize("attn", [True, False])
def test_activation_modes_ragged(attn, mode, tol):
    """hi + lo activations (~16 significant bits) and f16 activations (11 bits): the
    projections see the activations at that precision, so the forward is several times
    closer to the float64 oracle than with plain bf16 operands (8 significant bits)."""
    need_gpu()
    wl = Workload("ragged_act", 14, 300, 5, 50_000, 250, 24, 40, 3, 40, attn, "bf16", "sum", 1.1, act_mode=mode)
    run_full_compare(wl, fwd_tol=tol)


@pytest.mark.parametrize("rank,batch", [(296, 77), (600, 37)])
def test_attention_multiwave_ragged(rank, batch):
    """Ranks above 256 split one sample's rows over 2 or 4 waves of a workgroup (the
    backward adds their column sums in wave order); odd batches leave idle waves in
    the last workgroup, and ranks that are no multiple of 32 leave padded keys."""
    need_gpu()
    wl = Workload("multiwave", 15, batch, 4, 20_000, 150, 16, 64, 2, rank, True, "bf16", "sum", 1.1)
    run_full_compare(wl)


@pytest.mark.parametrize("tau,beta", [(1.0, 1.0), (0.25, 0.5), (4.0, 0.0)])
def test_parallel_branches_ragged(tau, beta):
    """Plain and attention low-rank cross nets with their own weights: batch 300, d = 160,
    r = 40 (no tile multiples), two layers."""
    need_gpu()
    wl = Workload("parallel", 16, 300, 5, 50_000, 250, 24, 40, 2, 40, True, "bf16", "sum", 1.1, temperature=tau,
                  parallel=True)
    run_full_compare(wl.with_(skip_beta=beta))


def test_parallel_branches_fp32_ragged():
    need_gpu()
    wl = Workload("parallel32", 17, 130, 3, 10_000, 100, 16, 12, 3, 20, True, "f32", "mul", 1.1, parallel=True)
    run_full_compare(wl)


def test_parallel_branches_small_full_batch_sampled():
    need_gpu()
    wl = WORKLOADS["small"].with_(parallel=True)
    rows = sample_rows(wl.batch, 24)
    run_full_compare(wl, grad_rows=rows, fwd_rows=rows)


def test_fp32_attention_ragged():
    need_gpu()
    wl = Workload("ragged32", 12, 130, 3, 10_000, 100, 16, 12, 3, 20, True, "f32", "mul", 1.1)
    run_full_compare(wl)


@pytest.mark.parametrize("name", ["feed", "multihot", "large"])
def test_full_batch_whole_tiles(name):
    """Whole 256-row tiles (the first, one in the middle, the last) at the full batch,
    with a dense upstream gradient on them: every element of those tiles of x_L and
    grad_x0 and of every weight gradient is compared."""
    need_gpu()
    wl = WORKLOADS[name]
    rows = tile_rows(wl.batch)
    run_full_compare(wl, grad_rows=rows, fwd_rows=rows, pool=True)


def test_small_forward_all_rows_and_gradient_tiles():
    """The small workload's forward on all 4096 rows; its gradients on three whole tiles."""
    need_gpu()
    wl = WORKLOADS["small"]
    run_full_compare(wl, grad_rows=tile_rows(wl.batch), fwd_rows=np.arange(wl.batch), pool=True)


@pytest.mark.parametrize("name,k", [("small", 24), ("feed", 12), ("multihot", 12), ("large", 40)])
def test_full_batch_sampled(name, k):
    """Large samples 40 rows: its 6-layer attention stack ends near one-hot (|logits| ~ 130),
    so single rows' gradients are sensitive to bf16 operand rounding (per-row errors 0.01-0.13
    measured); weight gradients summed over tens of rows average this out (0.03-0.043 on 48 rows)."""
    need_gpu()
    wl = WORKLOADS[name]
    rows = sample_rows(wl.batch, k)
    run_full_compare(wl, grad_rows=rows, fwd_rows=rows)


def test_small_rank_order_ids_full_batch():
    need_gpu()
    wl = WORKLOADS["small"]
    rows = sample_rows(wl.batch, 8)
    run_full_compare(wl, grad_rows=rows, fwd_rows=rows, id_mode="rank")


def test_zero_query_gives_uniform_attention():
    """Query weights zero => A = 11^T / r: the GPU forward matches the oracle, and the
    oracle in turn matches a dense DCNv2 with W = U (beta I + alpha/r 11^T) V^T."""
    need_gpu()
    wl = Workload("uniform", 13, 256, 4, 10_000, 100, 16, 64, 2, 32, True, "bf16", "sum", 1.1)
    inp = make_inputs(wl, bias_std=0.1)
    r = wl.rank
    for w in inp["w_down"]:
        w[r:2 * r] = 0
    db = DeviceBatch(wl, inp)
    db.gather()
    db.forward()
    x0 = oracle_x0(wl, inp)
    W, U, b = host_weights(inp)
    M = wl.beta * np.eye(r) + wl.alpha / r * np.ones((r, r))
    x = x0.astype(np.float64)
    for Wl, Ul, bl in zip(W, U, b):
        x = x0 * (x @ (Ul @ M @ Wl[:r]).T + bl) + x
    assert relerr(to_np(db.x_out), x) <= FWD_TOL["bf16"]


def test_deterministic_rerun():
    need_gpu()
    wl = WORKLOADS["small"].with_(batch=1024)
    inp = make_inputs(wl, bias_std=0.1)
    outs = []
    for _ in range(2):
        db = DeviceBatch(wl, inp)
        db.gather()
        db.forward()
        db.backward()
        torch.cuda.synchronize()
        outs.append([db.x_out.cpu(), db.grad_x0.cpu()] + [t.cpu() for t in db.g_w_down + db.g_u + db.g_bias])
    for a, b in zip(*outs):
        assert torch.equal(a.view(torch.uint8) if a.dtype == torch.bfloat16 else a, b.view(torch.uint8)
                           if b.dtype == torch.bfloat16 else b)


def test_batch_zero_and_batch_one():
    need_gpu()
    wl = WORKLOADS["small"].with_(batch=1)
    run_full_compare(wl)
    inp = make_inputs(WORKLOADS["small"].with_(batch=4), bias_std=0.1)
    db = DeviceBatch(WORKLOADS["small"].with_(batch=4), inp)
    db.B = 0
    db.gather()
    db.forward()
    db.backward()
    torch.cuda.synchronize()
    for t in db.g_w_down + db.g_u + db.g_bias:
        assert not torch.any(t)


def test_f16_activation_overflow_is_reported():
    """Activation mode 2 keeps x_l (l >= 1) in f16: a dense input of 7e4 (exact in bf16)
    makes x_1 exceed the f16 range, and the forward reports RDCN_ERR_RANGE through the
    device error word (read and cleared by rdcn_check_device_errors); a normal batch on
    the same handle then reads as RDCN_OK."""
    need_gpu()
    from paper_2402_06859_amd import rdcn
    wl = Workload("ovf_f16", 15, 64, 3, 5_000, 80, 16, 24, 2, 16, False, "bf16", "sum", 1.1, act_mode="f16")
    inp = make_inputs(wl)
    big = dict(inp, dense=torch.full_like(inp["dense"], 7.0e4))
    db = DeviceBatch(wl, big)
    db.gather()
    db.forward()
    torch.cuda.synchronize()
    assert db.lib.check_device_errors() == rdcn.RDCN_ERR_RANGE
    assert db.lib.check_device_errors() == rdcn.RDCN_OK  # cleared by the read
    db2 = DeviceBatch(wl, inp)
    db2.gather()
    db2.forward()
    torch.cuda.synchronize()
    assert db2.lib.check_device_errors() == rdcn.RDCN_OK
