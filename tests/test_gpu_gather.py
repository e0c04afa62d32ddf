"""GPU gather (qr_embed_gather) vs the oracle: bit-exact x0 on every workload
at its full batch, both combines, both id widths, rank-order (hot-row) ids,
bags including empty ones, and the out-of-range id flag."""
import numpy as np
import pytest
import torch

from gpu_helpers import bf16_bits, need_gpu, oracle_x0
from paper_2402_06859_amd import rdcn
from paper_2402_06859_amd.synth import WORKLOADS, make_inputs

pytestmark = pytest.mark.gpu


def run_gather(wl, inp, id_type="i64"):
    lib = rdcn.Rdcn(rdcn.config_for(wl, inp["batch"], id_type))
    dev = torch.device("cuda")
    ids = inp["ids"] if id_type == "i64" else inp["ids"].to(torch.int32)
    ids = ids.contiguous().to(dev)
    offs = None if inp["offsets"] is None else inp["offsets"].to(dev)
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    x0 = torch.full((inp["batch"], wl.d), float("nan"), dtype=dt, device=dev)
    lib.qr_embed_gather(inp["batch"], ids, offs, inp["q_tables"].to(dev), inp["r_tables"].to(dev),
                        inp["dense"].to(dev), x0)
    status = lib.check_device_errors()
    return x0.cpu(), status


def assert_bitexact(wl, x0_gpu, x0_ref):
    if wl.dtype == "bf16":
        ref_bits = torch.from_numpy(x0_ref).to(torch.bfloat16).view(torch.int16).numpy()
        got = bf16_bits(x0_gpu)
    else:
        ref_bits = x0_ref.view(np.int32)
        got = x0_gpu.numpy().view(np.int32)
    mism = np.argwhere(got != ref_bits)
    assert mism.size == 0, "first mismatches at %s" % mism[:5].tolist()


@pytest.mark.parametrize("name", ["tiny", "small", "feed", "multihot", "large"])
def test_gather_bitexact_full_batch(name):
    need_gpu()
    wl = WORKLOADS[name]
    inp = make_inputs(wl, with_weights=False, with_grad=False)
    print("gather", name, "B", inp["batch"], flush=True)
    x0, status = run_gather(wl, inp)
    assert status == rdcn.RDCN_OK
    assert_bitexact(wl, x0, oracle_x0(wl, inp))


@pytest.mark.parametrize("name,combine,id_type,mode", [
    ("small", "mul", "i32", "rank"), ("small", "sum", "i32", "rank"), ("tiny", "sum", "i64", "rank"),
    ("multihot", "mul", "i32", "scatter")])
def test_gather_variants(name, combine, id_type, mode):
    need_gpu()
    wl = WORKLOADS[name].with_(combine=combine)
    if name == "multihot":
        wl = wl.with_(batch=512)
    inp = make_inputs(wl, id_mode=mode, with_weights=False, with_grad=False)
    x0, status = run_gather(wl, inp, id_type)
    assert status == rdcn.RDCN_OK
    assert_bitexact(wl, x0, oracle_x0(wl, inp))


@pytest.mark.parametrize("batch,F,D,Nd,dtype,multi_hot", [
    # 3 column blocks (two holding embedding columns, one dense-only), 37 row groups:
    # both item counts leave remainders after the split over the 8 XCDs
    (587, 10, 64, 896, "bf16", False),
    (587, 10, 64, 896, "bf16", True),
    # one column block, float storage, a ragged last column block of 13 vectors
    (1001, 3, 4, 40, "f32", False),
    # more than 65535 row groups of 16 rows: the row groups are walked grid-stride
    (1_100_000, 2, 8, 8, "bf16", False),
    (1_050_001, 1, 4, 4, "f32", True),
])
def test_gather_grid_shapes(batch, F, D, Nd, dtype, multi_hot):
    """x0 bit-exact on shapes chosen for the launch's block mapping rather than for a
    workload: remainders in the per-XCD split, a dense-only column block, and batches
    past the grid's row-group limit."""
    need_gpu()
    wl = WORKLOADS["tiny"].with_(batch=batch, num_cat=F, emb_dim=D, num_dense=Nd, dtype=dtype,
                                 multi_hot=multi_hot, bag_mean=3.0, bag_max=8)
    inp = make_inputs(wl, with_weights=False, with_grad=False)
    print("gather grid shape B %d F %d D %d Nd %d %s bags %s" % (batch, F, D, Nd, dtype, multi_hot), flush=True)
    x0, status = run_gather(wl, inp)
    assert status == rdcn.RDCN_OK
    assert_bitexact(wl, x0, oracle_x0(wl, inp))


# Row 0 of both tables: per column, a pair whose combine rounds to bf16 at an edge.
# sum: ties to even (down and up), a tie at the largest finite value (to infinity, both
# signs), a tie at 3 (stays), values below and above half an ulp. mul: ties to even in the normal
# range (down, up), products below the float normal range that round to a bf16 denormal
# or to zero (ties to even, signed zero), above half an ulp, and a float overflow.
_BF16_MAX = (2.0 - 2.0 ** -7) * 2.0 ** 127
_EDGES = {
    "sum": ([1.0, 1 + 2 ** -7, _BF16_MAX, -_BF16_MAX, 3.0, -(1 + 2 ** -7), 1.0, 2.0],
            [2 ** -8, 2 ** -8, 2.0 ** 119, -2.0 ** 119, 2 ** -7, -2 ** -8, 2 ** -9, 3 * 2 ** -8]),
    "mul": ([1 + 8 * 2 ** -7, 1 + 2 ** -7, 2.0 ** -67, 1.5 * 2.0 ** -66, 1.25 * 2.0 ** -65, 1.75 * 2.0 ** -66,
             -(2.0 ** -67), (2 - 2 ** -7) * 2.0 ** 64],
            [1 + 8 * 2 ** -7, 1 + 64 * 2 ** -7, 2.0 ** -67, 2.0 ** -67, 2.0 ** -67, 2.0 ** -67, 2.0 ** -67,
             (2 - 2 ** -7) * 2.0 ** 63]),
}


@pytest.mark.parametrize("combine", ["sum", "mul"])
def test_gather_bf16_rounding_edges(combine):
    """x0 bit-exact where rounding the float combine to bf16 is decided by a tie, by a
    result below the float normal range or by overflow: the conversion every bf16 output
    of the library goes through."""
    need_gpu()
    wl = WORKLOADS["tiny"].with_(dtype="bf16", combine=combine, batch=40, num_cat=2, emb_dim=8, num_dense=8,
                                 vocab=256, table_rows=16)
    inp = make_inputs(wl, with_weights=False, with_grad=False)
    qv, rv = _EDGES[combine]
    for t, vals in (("q_tables", qv), ("r_tables", rv)):
        tab = inp[t].float()
        tab[:, 0, :] = torch.tensor(vals, dtype=torch.float32)
        assert torch.equal(tab[:, 0, :].to(torch.bfloat16).float(), tab[:, 0, :]), "edge values are bf16 values"
        inp[t] = tab.to(torch.bfloat16)
    inp["ids"][::2, :] = 0  # even rows: id 0 = (quotient row 0, remainder row 0) in both features
    x0, status = run_gather(wl, inp)
    assert status == rdcn.RDCN_OK
    ref = oracle_x0(wl, inp)
    assert_bitexact(wl, x0, ref)
    # the oracle's values on the edge rows are the ones intended
    got = torch.from_numpy(np.ascontiguousarray(ref[0, :8])).to(torch.bfloat16).view(torch.int16).numpy().astype(np.int64) & 0xffff
    want = {"sum": [0x3F80, 0x3F82, 0x7F80, 0xFF80, 0x4040, 0xBF82, 0x3F80, 0x4001],
            "mul": [0x3F90, 0x3FC2, 0x0000, 0x0002, 0x0002, 0x0002, 0x8000, 0x7F80]}[combine]
    assert got.tolist() == want, [hex(v) for v in got.tolist()]


def test_gather_ragged_batch_and_bags_with_empty_and_bad_ids():
    need_gpu()
    wl = WORKLOADS["multihot"].with_(batch=37, num_cat=3, num_dense=8)
    inp = make_inputs(wl, with_weights=False, with_grad=False)
    # empty every 5th bag; put one out-of-range id into bag 7
    offs = inp["offsets"].numpy()
    ids = inp["ids"].numpy()
    lens = np.diff(offs)
    lens[::5] = 0
    new_offs = np.zeros_like(offs)
    np.cumsum(lens, out=new_offs[1:])
    new_ids = np.concatenate([ids[offs[i]:offs[i] + lens[i]] for i in range(len(lens))])
    new_ids[new_offs[7]] = wl.vocab + 5
    inp["offsets"] = torch.from_numpy(new_offs)
    inp["ids"] = torch.from_numpy(new_ids)
    x0, status = run_gather(wl, inp)
    assert status == rdcn.RDCN_ERR_INDEX
    from oracle import gather
    ref, bad = gather(37, 3, wl.emb_dim, 8, wl.vocab, wl.table_rows, wl.table_rows, wl.combine, True,
                      inp["ids"], inp["offsets"], inp["q_tables"], inp["r_tables"], inp["dense"])
    assert bad == 1
    assert_bitexact(wl, x0, ref)


def test_gather_out_of_range_single_hot_flag_clears():
    need_gpu()
    wl = WORKLOADS["tiny"]
    inp = make_inputs(wl, with_weights=False, with_grad=False)
    inp["ids"][3, 2] = -1
    _, status = run_gather(wl, inp)
    assert status == rdcn.RDCN_ERR_INDEX
    inp["ids"][3, 2] = 0
    _, status = run_gather(wl, inp)
    assert status == rdcn.RDCN_OK
