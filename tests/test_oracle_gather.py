"""Pins for the oracle's gather (QR combine, bag pooling, concat with dense).

Lookup is checked against an independent formulation: one-hot selection
matrices times the tables in float64 (the 'sparse one-hot input replaced by
embedding look-ups' of section 'Residual DCN'). Rounding to bfloat16 is checked
against torch's conversion (round to nearest even).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2402_06859_amd.synth import WORKLOADS, make_inputs


def onehot(idx, n):
    P = np.zeros((idx.size, n))
    P[np.arange(idx.size), idx] = 1.0
    return P


def test_round_bf16_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(100_000).astype(np.float32) * np.float32(10.0) ** rng.integers(-30, 30, 100_000),
        np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 0.0, -0.0, np.inf, -np.inf,
                  3.3895e38, 1e-40, -1e-42], np.float32)])
    x = x.astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).float().numpy()
    got = oracle.round_bf16(x)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_round_f16_against_the_binary16_format():
    """Values fixed by the binary16 format itself (11 significant bits, exponents
    -14 .. 15, subnormals down to 2^-24, round to nearest with ties to even), then a
    sweep against torch's half conversion."""
    cases = [(1.0 / 3.0, 1365 / 4096),               # 1.0101010101 x 2^-2, next bit 0
             (0.1, 1638 / 16384), (-0.1, -1638 / 16384),
             (1 + 2 ** -11, 1.0),                    # tie, even neighbour 1
             (1 + 3 * 2 ** -11, 1 + 2 ** -9),        # tie, even neighbour 1 + 2^-9
             (1 + 2 ** -11 + 2 ** -20, 1 + 2 ** -10),  # just above the tie
             (65504.0, 65504.0), (65519.0, 65504.0), (65520.0, np.inf), (-70000.0, -np.inf),
             (2.0 ** -14, 2.0 ** -14), (2.0 ** -24, 2.0 ** -24), (2.0 ** -25, 0.0),
             (3 * 2.0 ** -26, 2.0 ** -24), (5 * 2.0 ** -25, 2 * 2.0 ** -24)]
    x = np.array([c[0] for c in cases], np.float32)
    want = np.array([c[1] for c in cases], np.float32)
    assert np.array_equal(oracle.round_f16(x), want)
    rng = np.random.default_rng(1)
    y = (rng.standard_normal(100_000) * 10.0 ** rng.integers(-9, 6, 100_000)).astype(np.float32)
    ref = torch.from_numpy(y).to(torch.float16).float().numpy()
    assert np.array_equal(oracle.round_f16(y).view(np.uint32), ref.view(np.uint32))


def test_gather_tiny_mul_vs_onehot():
    wl = WORKLOADS["tiny"]
    inp = make_inputs(wl, with_weights=False, with_grad=False)
    B, F, D, Nd, V, m = wl.batch, wl.num_cat, wl.emb_dim, wl.num_dense, wl.vocab, wl.table_rows
    ids = inp["ids"].numpy()
    qt, rt, dense = (inp[k].float().numpy() for k in ("q_tables", "r_tables", "dense"))
    x0, bad = oracle.gather(B, F, D, Nd, V, m, m, "mul", False, ids, None, qt, rt, dense)
    assert bad == 0
    for f in range(F):
        Pq = onehot(ids[:, f] // m, m)
        Pr = onehot(ids[:, f] % m, m)
        # float64 product of two floats is exact; one rounding to float32
        ref = ((Pq @ qt[f].astype(np.float64)) * (Pr @ rt[f].astype(np.float64))).astype(np.float32)
        assert np.array_equal(x0[:, f * D:(f + 1) * D], ref)
    assert np.array_equal(x0[:, F * D:], dense)


def test_gather_sum_bf16_matches_torch_add():
    wl = WORKLOADS["small"].with_(batch=256)
    inp = make_inputs(wl, with_weights=False, with_grad=False)
    B, F, D, Nd, V, m = 256, wl.num_cat, wl.emb_dim, wl.num_dense, wl.vocab, wl.table_rows
    ids = inp["ids"].numpy()
    qt, rt = inp["q_tables"].float(), inp["r_tables"].float()
    x0, bad = oracle.gather(B, F, D, Nd, V, m, m, "sum", True, ids, None, qt, rt, inp["dense"])
    assert bad == 0
    for f in (0, 17, F - 1):
        q = qt[f][torch.from_numpy(ids[:, f] // m)]
        r = rt[f][torch.from_numpy(ids[:, f] % m)]
        ref = (q + r).to(torch.bfloat16).float().numpy()
        assert np.array_equal(x0[:, f * D:(f + 1) * D].view(np.uint32), ref.view(np.uint32))
    assert np.array_equal(x0[:, F * D:], inp["dense"].float().numpy())


@pytest.mark.parametrize("combine", ["sum", "mul"])
def test_gather_bags_vs_count_matrix(combine):
    wl = WORKLOADS["multihot"].with_(batch=64, num_cat=5, combine=combine)
    inp = make_inputs(wl, with_weights=False, with_grad=False)
    B, F, D, Nd, V, m = 64, 5, wl.emb_dim, wl.num_dense, wl.vocab, wl.table_rows
    ids, offs = inp["ids"].numpy(), inp["offsets"].numpy()
    qt, rt = inp["q_tables"].float().numpy(), inp["r_tables"].float().numpy()
    x32, bad = oracle.gather(B, F, D, Nd, V, m, m, combine, False, ids, offs, qt, rt, inp["dense"])
    xbf, _ = oracle.gather(B, F, D, Nd, V, m, m, combine, True, ids, offs, qt, rt, inp["dense"])
    assert bad == 0
    u = 2.0 ** -24
    for b in range(B):
        for f in range(F):
            s, e = offs[b * F + f], offs[b * F + f + 1]
            q = qt[f][ids[s:e] // m].astype(np.float64)
            r = rt[f][ids[s:e] % m].astype(np.float64)
            terms = q * r if combine == "mul" else q + r
            exact = terms.sum(0)
            # sequential float32 summation bound plus one rounding of each term
            bound = (e - s + 1) * u * np.abs(terms).sum(0) + 1e-30
            got = x32[b, f * D:(f + 1) * D]
            assert np.all(np.abs(got - exact) <= bound)
            # bfloat16 result is the RNE rounding of the float32 result
            assert np.array_equal(xbf[b, f * D:(f + 1) * D], oracle.round_bf16(got))


def test_gather_bag_special_cases():
    F, D, V, m = 2, 8, 100, 10
    rng = np.random.default_rng(1)
    qt = rng.standard_normal((F, m, D)).astype(np.float32)
    rt = rng.standard_normal((F, m, D)).astype(np.float32)
    # one bag of length 1, one empty bag, one bag with an out-of-range id
    ids = np.array([37, 5, 200, 42], dtype=np.int64)
    offs = np.array([0, 1, 1, 2, 4], dtype=np.int64)  # B = 2: bags (0,0)=[37], (0,1)=[], (1,0)=[5], (1,1)=[200, 42]
    x0, bad = oracle.gather(2, F, D, 0, V, m, m, "sum", False, ids, offs, qt, rt, np.zeros((2, 0), np.float32))
    assert bad == 1
    single, _ = oracle.gather(1, 1, D, 0, V, m, m, "sum", False, np.array([[37]]), None, qt[:1], rt[:1],
                              np.zeros((1, 0), np.float32))
    assert np.array_equal(x0[0, :D], single[0])
    assert np.all(x0[0, D:] == 0) and not np.any(np.signbit(x0[0, D:]))
    assert np.array_equal(x0[1, D:], qt[1, 4] + rt[1, 2])  # 42 -> (4, 2); the bad id adds nothing


def test_gather_signed_zero_pooling():
    """Pooling starts from the first element, so a bag of -0.0 terms stays -0.0."""
    D, m = 4, 4
    qt = np.full((1, m, D), -0.0, np.float32)
    rt = np.ones((1, m, D), np.float32)
    ids = np.array([1, 2, 3], dtype=np.int64)
    offs = np.array([0, 3], dtype=np.int64)
    x0, _ = oracle.gather(1, 1, D, 0, 16, m, m, "mul", True, ids, offs, qt, rt, np.zeros((1, 0), np.float32))
    assert np.all(x0 == 0) and np.all(np.signbit(x0))
