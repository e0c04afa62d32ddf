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


def unreached(wl, inp):
    """Rows of the quotient / remainder tables that no valid id reaches, [F, rows] masks."""
    F, V, m = wl.num_cat, wl.vocab, wl.table_rows
    ids = inp["ids"].numpy().astype(np.int64)
    if inp["offsets"] is None:
        feat = np.tile(np.arange(F), inp["batch"])
        ids = ids.reshape(-1)
    else:
        lens = np.diff(inp["offsets"].numpy())
        feat = np.repeat(np.tile(np.arange(F), inp["batch"]), lens)
    ok = (ids >= 0) & (ids < V)
    q = np.ones((F, m), dtype=bool)
    r = np.ones((F, m), dtype=bool)
    q[feat[ok], ids[ok] // m] = False
    r[feat[ok], ids[ok] % m] = False
    return q, r


def assert_unreached_zero(wl, inp, gq, gr):
    """Rows that no id reaches stay exactly zero (a reached row may still sum to 0)."""
    uq, ur = unreached(wl, inp)
    assert not np.any(gq.numpy()[uq]) and not np.any(gr.numpy()[ur])


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
    assert_unreached_zero(wl, inp, gq, gr)


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


def test_embed_backward_sort_path_large_tables():
    """Tables of more than 16384 rows take the keys / radix sort / segmented-reduce path
    (scratch > 0); tables of at most 16384 rows the one-kernel path (no scratch)."""
    need_gpu()
    wl = WORKLOADS["small"].with_(batch=2048, vocab=400_000_000, table_rows=20_000)
    inp = make_inputs(wl, id_mode="rank", with_weights=False, with_grad=False)
    lib = rdcn.Rdcn(rdcn.config_for(wl, inp["batch"]))
    assert lib.embed_backward_workspace(inp["batch"], inp["ids"].numel()) > 0
    small = rdcn.Rdcn(rdcn.config_for(WORKLOADS["small"], 4096))
    assert small.embed_backward_workspace(4096, 4096 * 50) == 0
    gx0 = grad_x0_like(wl, inp["batch"], 9)
    print("embed_bwd sort path", flush=True)
    gq, gr, status = run(wl, inp, gx0)
    assert status == rdcn.RDCN_OK
    rq, rr, _ = ref(wl, inp, gx0)
    assert max(relerr(gq.numpy(), rq), relerr(gr.numpy(), rr)) <= 1e-5


@pytest.mark.parametrize("batch,mode", [(9000, "rank"), (4097, "scatter"), (1, "rank")])
def test_embed_backward_single_hot_chunks(batch, mode):
    """Single-hot batches over several 4096-occurrence chunks, ragged last chunk, and one
    sample; rank-order ids put most occurrences on one quotient row (a segment across
    all four wave parts of every chunk)."""
    need_gpu()
    wl = WORKLOADS["small"].with_(batch=batch, num_cat=5)
    inp = make_inputs(wl, id_mode=mode, with_weights=False, with_grad=False)
    gx0 = grad_x0_like(wl, batch, 10)
    print("embed_bwd single-hot", batch, mode, flush=True)
    gq, gr, status = run(wl, inp, gx0)
    assert status == rdcn.RDCN_OK
    rq, rr, _ = ref(wl, inp, gx0)
    assert max(relerr(gq.numpy(), rq), relerr(gr.numpy(), rr)) <= 1e-5
    assert_unreached_zero(wl, inp, gq, gr)


@pytest.mark.parametrize("F,combine", [(3, "sum"), (3, "mul"), (64, "sum"), (64, "mul"), (120, "sum")])
def test_embed_backward_bag_edges(F, combine):
    """Bags: empty bags, a bag longer than a chunk, bags of one, and a hot id that takes
    half of all occurrences; both combines. The feature count sets the slice count and
    so the kernel form: 3 features, slices of at most 1024 rows (4096-occurrence
    chunks); 64, slices of 1582 rows (8192-occurrence chunks with the sum combine, 4096
    with the product); 120, whole 3163-row tables."""
    need_gpu()
    B = 700
    wl = WORKLOADS["multihot"].with_(batch=B, num_cat=F, combine=combine, emb_dim=32, num_dense=16)
    inp = make_inputs(wl, with_weights=False, with_grad=False)
    rng = np.random.Generator(np.random.PCG64(11))
    lens = rng.integers(0, 12, size=(B, F))
    lens[rng.random((B, F)) < 0.2] = 0      # empty bags
    lens[5, 1] = 5000 if F < 64 else 9000   # longer than one chunk
    lens[600, 2] = 4500 if F < 64 else 8500
    lens[7, :] = 1
    offsets = np.zeros(B * F + 1, dtype=np.int64)
    np.cumsum(lens.reshape(-1), out=offsets[1:])
    nnz = int(offsets[-1])
    ids = rng.integers(0, wl.vocab, size=nnz)
    ids[rng.random(nnz) < 0.5] = 123_457   # hot id: one long segment per table
    inp["ids"] = torch.from_numpy(ids.astype(np.int64))
    inp["offsets"] = torch.from_numpy(offsets)
    gx0 = grad_x0_like(wl, B, 12)
    print("embed_bwd bag edges", F, combine, "nnz", nnz, flush=True)
    gq, gr, status = run(wl, inp, gx0)
    assert status == rdcn.RDCN_OK
    rq, rr, _ = ref(wl, inp, gx0)
    assert max(relerr(gq.numpy(), rq), relerr(gr.numpy(), rr)) <= 1e-5
    assert_unreached_zero(wl, inp, gq, gr)


@pytest.mark.parametrize("F,combine", [(3, "sum"), (64, "sum"), (64, "mul"), (120, "sum")])
def test_embed_backward_bag_passes(F, combine):
    """Bags over several passes of 1024 bags: a pass that is not the batch's last takes
    only the leading bags that fill whole chunks, and the next pass starts after them.
    Covered: a pass that starts with a bag longer than a chunk (only that bag is taken:
    feature 1 with 8192-occurrence chunks, feature 2 with 4096), empty bags at the cuts,
    bags that span chunk boundaries, a hot id; compared with the oracle and rerun
    bitwise."""
    need_gpu()
    B = 2600
    wl = WORKLOADS["multihot"].with_(batch=B, num_cat=F, combine=combine, emb_dim=32, num_dense=16)
    inp = make_inputs(wl, with_weights=False, with_grad=False)
    rng = np.random.Generator(np.random.PCG64(17))
    lens = rng.integers(0, 12, size=(B, F))
    lens[rng.random((B, F)) < 0.2] = 0      # empty bags
    lens[1024, 1 % F] = 9000                 # first bag of the second pass, longer than any chunk
    if F > 2:
        lens[1025:2048, 2] = 0               # feature 2's second pass: one long bag and a few short ones
        lens[1025:2048:100, 2] = 3
        lens[1024, 2] = 5000
    offsets = np.zeros(B * F + 1, dtype=np.int64)
    np.cumsum(lens.reshape(-1), out=offsets[1:])
    nnz = int(offsets[-1])
    ids = rng.integers(0, wl.vocab, size=nnz)
    ids[rng.random(nnz) < 0.5] = 123_457    # hot id: one long segment per table
    inp["ids"] = torch.from_numpy(ids.astype(np.int64))
    inp["offsets"] = torch.from_numpy(offsets)
    gx0 = grad_x0_like(wl, B, 19)
    print("embed_bwd bag passes", F, combine, "nnz", nnz, flush=True)
    gq, gr, status = run(wl, inp, gx0)
    assert status == rdcn.RDCN_OK
    rq, rr, _ = ref(wl, inp, gx0)
    assert max(relerr(gq.numpy(), rq), relerr(gr.numpy(), rr)) <= 1e-5
    assert_unreached_zero(wl, inp, gq, gr)
    gq2, gr2, _ = run(wl, inp, gx0)
    assert torch.equal(gq, gq2) and torch.equal(gr, gr2)


@pytest.mark.parametrize("D,dtype", [(4, "f32"), (48, "bf16"), (256, "bf16")])
def test_embed_backward_widths(D, dtype):
    """Table widths from one column group to 256 (one pair per step)."""
    need_gpu()
    wl = WORKLOADS["tiny"].with_(emb_dim=D, combine="sum", dtype=dtype)
    inp = make_inputs(wl, id_mode="rank", with_weights=False, with_grad=False)
    gx0 = grad_x0_like(wl, inp["batch"], 13)
    print("embed_bwd width", D, flush=True)
    gq, gr, status = run(wl, inp, gx0)
    assert status == rdcn.RDCN_OK
    rq, rr, _ = ref(wl, inp, gx0)
    assert max(relerr(gq.numpy(), rq), relerr(gr.numpy(), rr)) <= 1e-5
