"""GPU middle-max 8-bit table quantization (qr_quantize_tables) and the serving
gather from quantized tables (qr_embed_gather_q8) vs the oracle: codes, row
parameters and x0 bit-exact on every workload at its full batch, both combines,
bags with empty bags and a bad id, and rows that are constant, hold signed
zeros or put values on rounding ties."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import bf16_bits, need_gpu
from paper_2402_06859_amd import rdcn
from paper_2402_06859_amd.synth import WORKLOADS, make_inputs

pytestmark = pytest.mark.gpu


def quantize_gpu(lib, tables, D):
    rows = tables.numel() // D
    dev = torch.device("cuda")
    codes = torch.empty((rows, D), dtype=torch.int8, device=dev)
    params = torch.empty((rows, 2), dtype=torch.float32, device=dev)
    lib.qr_quantize_tables(rows, tables.contiguous().to(dev), codes, params)
    torch.cuda.synchronize()
    return codes, params


def check_quantize(lib, tables, D):
    codes, params = quantize_gpu(lib, tables, D)
    ref_c, ref_p = oracle.quantize_rows(tables.float().numpy().reshape(-1, D))
    got_c, got_p = codes.cpu().numpy(), params.cpu().numpy()
    bad = np.argwhere(got_c != ref_c)
    assert bad.size == 0, "code mismatches at %s" % bad[:5].tolist()
    assert np.array_equal(got_p.view(np.uint32), ref_p.view(np.uint32))
    return codes, params


def gather_q8(wl, inp, id_type="i64"):
    B = inp["batch"]
    F, D, m = wl.num_cat, wl.emb_dim, wl.table_rows
    lib = rdcn.Rdcn(rdcn.config_for(wl, B, id_type))
    qc, qp = check_quantize(lib, inp["q_tables"], D)
    rc, rp = check_quantize(lib, inp["r_tables"], D)
    dev = torch.device("cuda")
    ids = (inp["ids"] if id_type == "i64" else inp["ids"].to(torch.int32)).contiguous().to(dev)
    offs = None if inp["offsets"] is None else inp["offsets"].to(dev)
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    x0 = torch.full((B, wl.d), float("nan"), dtype=dt, device=dev)
    lib.qr_embed_gather_q8(B, ids, offs, qc, qp, rc, rp, inp["dense"].to(dev), x0)
    status = lib.check_device_errors()
    ref, nbad = oracle.gather_q8(B, F, D, wl.num_dense, wl.vocab, m, m, wl.combine, wl.dtype == "bf16", inp["ids"],
                                 inp["offsets"], qc.cpu().numpy(), qp.cpu().numpy(), rc.cpu().numpy(),
                                 rp.cpu().numpy(), inp["dense"])
    if wl.dtype == "bf16":
        ref_bits = torch.from_numpy(ref).to(torch.bfloat16).view(torch.int16).numpy()
        got = bf16_bits(x0)
    else:
        ref_bits, got = ref.view(np.int32), x0.cpu().numpy().view(np.int32)
    mism = np.argwhere(got != ref_bits)
    assert mism.size == 0, "first x0 mismatches at %s" % mism[:5].tolist()
    return status, nbad


@pytest.mark.parametrize("name", ["tiny", "small", "feed", "multihot", "large"])
def test_quantized_gather_bitexact_full_batch(name):
    need_gpu()
    wl = WORKLOADS[name]
    inp = make_inputs(wl, with_weights=False, with_grad=False)
    print("gather_q8", name, "B", inp["batch"], flush=True)
    status, nbad = gather_q8(wl, inp)
    assert status == rdcn.RDCN_OK and nbad == 0


@pytest.mark.parametrize("name,combine,id_type", [("small", "mul", "i32"), ("tiny", "sum", "i64"),
                                                  ("multihot", "mul", "i32")])
def test_quantized_gather_variants(name, combine, id_type):
    need_gpu()
    wl = WORKLOADS[name].with_(combine=combine)
    if name == "multihot":
        wl = wl.with_(batch=512)
    inp = make_inputs(wl, id_mode="rank", with_weights=False, with_grad=False)
    status, nbad = gather_q8(wl, inp, id_type)
    assert status == rdcn.RDCN_OK and nbad == 0


def test_quantized_gather_bags_empty_and_bad_id():
    need_gpu()
    wl = WORKLOADS["multihot"].with_(batch=37, num_cat=3, num_dense=8)
    inp = make_inputs(wl, with_weights=False, with_grad=False)
    offs, ids = inp["offsets"].numpy(), inp["ids"].numpy()
    lens = np.diff(offs)
    lens[::4] = 0
    new_offs = np.zeros_like(offs)
    np.cumsum(lens, out=new_offs[1:])
    new_ids = np.concatenate([ids[offs[i]:offs[i] + lens[i]] for i in range(len(lens))])
    new_ids[new_offs[9]] = -3
    inp["offsets"], inp["ids"] = torch.from_numpy(new_offs), torch.from_numpy(new_ids)
    status, nbad = gather_q8(wl, inp)
    assert status == rdcn.RDCN_ERR_INDEX and nbad == 1


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_quantize_special_rows(dtype):
    """Constant rows, signed zeros, exact grid rows with half-way values, one huge
    outlier, and a row whose values are all equal but one."""
    need_gpu()
    D = 16
    rows = [np.full(D, 0.75), np.zeros(D), np.where(np.arange(D) % 2 == 0, -0.0, 0.0),
            np.linspace(-128, 127, D), np.r_[np.arange(-8, 7) + 0.5, 127.0], np.r_[np.zeros(D - 1), 1e30],
            np.r_[np.full(D - 1, -1.0), 2.0]]
    rng = np.random.default_rng(1)
    rows += [rng.standard_normal(D) * s for s in (1e-30, 1e-3, 1.0, 1e3, 1e30)]
    x = torch.tensor(np.stack(rows), dtype=torch.float32)
    if dtype == "bf16":
        x = x.to(torch.bfloat16)
    wl = WORKLOADS["small" if dtype == "bf16" else "tiny"].with_(emb_dim=D)
    lib = rdcn.Rdcn(rdcn.config_for(wl, 16))
    check_quantize(lib, x, D)
