"""GPU embedding backward (qr_embed_backward) vs the oracle: both combines,
single-hot and bags, scattered and rank-order (hot-row) ids, full batches;
accumulation (+=), determinism (bitwise rerun), and bad ids skipped."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import GRAD_TOL, need_gpu, relerr, to_np
from paper_2402_06859_amd import rdcn
from paper_2402_06859_amd.synth import WORKLOADS, grad_x0_like, make_inputs

pytestmark = pytest.mark.gpu


def run(wl, inp, gx0, id_type="i64", reps=1):
    lib = rdcn.Rdcn(rdcn.config_for(wl, inp["batch"], id_type))
    dev = torch.device("cuda")
    ids = (inp["ids"] if id_type == "i64" else inp["ids"].to(torch.int32)).contiguous().to(dev)
    offs = None if inp["offsets"] is None else inp["offsets"].to(dev)
    nnz = int(inp["ids"].numel())
    qt, rt = inp["q_tables"].to(dev), inp["r_tables"].to(dev)
    gq = torch.zeros(qt.shape, dtype=torch.float32, device=dev)
    gr = torch.zeros(rt.shape, dtype=torch.float32, device=dev)
    scratch = torch.empty(lib.embed_backward_workspace(inp["batch"], nnz), dtype=torch.uint8, device=dev)
    g = gx0.to(dev)
    for _ in range(reps):
        lib.qr_embed_backward(inp["batch"], nnz, ids, offs, qt, rt, g, gq, gr, scratch)
    status = lib.check_device_errors()
    return gq.cpu(), gr.cpu(), status


def ref(wl, inp, gx0):
    gq, gr, bad = oracle.embed_backward(inp["batch"], wl.num_cat, wl.emb_dim, wl.num_dense, wl.vocab,
                                        wl.table_rows, wl.table_rows, wl.combine, inp["ids"], inp["offsets"],
                                        inp["q_tables"], inp["r_tables"], gx0.numpy())
    return gq, gr, bad


@pytest.mark.parametrize("name,mode", [("tiny", "scatter"), ("small", "scatter"), ("small", "rank"),
                                       ("feed", "scatter"), ("multihot", "scatter"), ("multihot", "rank"),
                                       ("large", "scatter")])
def test_embed_backward_full_batch(name, mode):
    need_gpu()
    wl = WORKLOADS[name]
    inp = make_inputs(wl, id_mode=mode, with_weights=False, with_grad=False)
    gx0 = grad_x0_like(wl, inp["batch"], 5)
    print("embed_bwd", name, mode, "nnz", inp["ids"].numel(), flush=True)
    gq, gr, status = run(wl, inp, gx0)
    assert status == rdcn.RDCN_OK
    rq, rr, _ = ref(wl, inp, gx0)
    e = (relerr(gq.numpy(), rq), relerr(gr.numpy(), rr))
    print("rel err", e, flush=True)
    tol = 1e-5 if wl.dtype == "f32" else 1e-5  # float sums of float inputs: only summation rounding differs
    assert max(e) <= tol
    # rows that no id reaches stay exactly zero
    assert np.array_equal(gq.numpy() == 0, rq == 0) and np.array_equal(gr.numpy() == 0, rr == 0)


@pytest.mark.parametrize("name", ["small", "multihot"])
def test_embed_backward_mul_combine_i32(name):
    need_gpu()
    wl = WORKLOADS[name].with_(combine="mul")
    if name == "multihot":
        wl = wl.with_(batch=1024)
    inp = make_inputs(wl, with_weights=False, with_grad=False)
    gx0 = grad_x0_like(wl, inp["batch"], 6)
    gq, gr, status = run(wl, inp, gx0, id_type="i32")
    rq, rr, _ = ref(wl, inp, gx0)
    assert status == rdcn.RDCN_OK
    assert max(relerr(gq.numpy(), rq), relerr(gr.numpy(), rr)) <= 1e-5


def test_embed_backward_accumulates_and_is_deterministic():
    need_gpu()
    wl = WORKLOADS["multihot"].with_(batch=2048)
    inp = make_inputs(wl, id_mode="rank", with_weights=False, with_grad=False)
    gx0 = grad_x0_like(wl, inp["batch"], 7)
    gq1, gr1, _ = run(wl, inp, gx0)
    gq1b, gr1b, _ = run(wl, inp, gx0)
    assert torch.equal(gq1, gq1b) and torch.equal(gr1, gr1b)
    gq2, gr2, _ = run(wl, inp, gx0, reps=2)
    rq, rr, _ = ref(wl, inp, gx0)
    assert max(relerr(gq2.numpy(), 2 * rq), relerr(gr2.numpy(), 2 * rr)) <= 1e-5


def test_embed_backward_skips_bad_ids():
    need_gpu()
    wl = WORKLOADS["tiny"]
    inp = make_inputs(wl, with_weights=False, with_grad=False)
    inp["ids"][10, 1] = wl.vocab
    inp["ids"][11, 0] = -3
    gx0 = grad_x0_like(wl, inp["batch"], 8)
    gq, gr, _ = run(wl, inp, gx0)
    rq, rr, bad = ref(wl, inp, gx0)
    assert bad == 2
    assert max(relerr(gq.numpy(), rq), relerr(gr.numpy(), rr)) <= 1e-5
