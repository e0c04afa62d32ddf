"""Pins for the oracle's middle-max 8-bit row-wise table quantization and the
serving gather from quantized tables (section 'Embedding Table Quantization').

What fixes the oracle here, independently of its own code:
  - exact cases: a row spanning [-128, 127] has middle 0 and scale 1, so codes
    are the values themselves (half-way values tie to even);
  - the definition in exact rational arithmetic (fractions), rounded half to
    even, on random rows: the float pipeline must agree except within float
    rounding of a tie;
  - the ends of the range: the row maximum maps to 127 and the minimum to -128
    (a swapped 2^(bits-1) / 2^(bits-1) - 1 weight or a min-max zero point moves
    one of them);
  - the relation to min-max quantization: middle = min + 128 * scale, so the
    middle-max code is the min-max code shifted by 128;
  - the dequantization error is at most half a step;
  - the paper's size example (golden fixture);
  - the quantized gather against one-hot selection products of the tables
    dequantized in float64 arithmetic.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2402_06859_amd.synth import WORKLOADS, make_inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def half_even(fr: Fraction) -> int:
    n = fr.numerator // fr.denominator
    rem = fr - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return n


def test_exact_grid_row():
    x = np.array([[-128.0, 127.0, 0.0, 5.0, -7.0, 2.5, 3.5, -0.5]], np.float32)
    codes, params = oracle.quantize_rows(x)
    assert params[0, 0] == 0.0 and params[0, 1] == 1.0
    assert codes[0].tolist() == [-128, 127, 0, 5, -7, 2, 4, 0]
    assert np.array_equal(oracle.dequantize_rows(codes, params)[0, :5], x[0, :5])


def test_matches_exact_rational_definition():
    rng = np.random.default_rng(11)
    x = (rng.standard_normal((200, 24)) * rng.uniform(0.01, 5, (200, 1))).astype(np.float32)
    codes, params = oracle.quantize_rows(x)
    near_tie = 0
    for i in range(x.shape[0]):
        row = [Fraction(float(v)) for v in x[i]]
        mn, mx = min(row), max(row)
        middle = (mx * 128 + mn * 127) / 255
        scale = (mx - mn) / 255
        # three roundings (mn*127, the sum, the division); the sum may cancel, so the
        # bound is relative to the terms, not to the middle itself
        terms = (128 * abs(float(mx)) + 127 * abs(float(mn))) / 255
        assert abs(float(middle) - params[i, 0]) <= 3 * 2.0 ** -24 * terms + np.spacing(np.float32(abs(float(middle))))
        assert abs(float(scale) - params[i, 1]) <= np.spacing(np.float32(float(scale)))
        for c, v in enumerate(row):
            q = (v - middle) / scale
            exact = half_even(q)
            if codes[i, c] != exact:
                # only where float rounding can move a value across a tie
                frac = q - (q.numerator // q.denominator)
                assert abs(float(frac) - 0.5) < 1e-4, (i, c, float(q), codes[i, c])
                near_tie += 1
    assert near_tie <= 5


def test_row_ends_map_to_code_range_ends():
    rng = np.random.default_rng(3)
    x = (rng.standard_normal((500, 32)) * 3).astype(np.float32)
    codes, params = oracle.quantize_rows(x)
    assert codes.min() >= -128 and codes.max() <= 127
    rows = np.arange(x.shape[0])
    assert np.all(codes[rows, x.argmax(1)] == 127)
    assert np.all(codes[rows, x.argmin(1)] == -128)
    # codes survive an int8 -> int32 -> int8 round trip unchanged (no 0..255 range)
    assert np.array_equal(codes.astype(np.int32).astype(np.int8), codes)


def test_relation_to_min_max_quantization():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((300, 16)).astype(np.float32)
    codes, params = oracle.quantize_rows(x)
    mn, mx = x.min(1).astype(np.float64), x.max(1).astype(np.float64)
    scale = (mx - mn) / 255
    minmax = np.rint((x - mn[:, None]) / scale[:, None])  # min-max codes in [0, 255]
    agree = (codes.astype(np.int64) + 128 == minmax)
    assert agree.mean() > 0.999  # both round the same real number; only ties in float may differ


def test_dequantization_error_at_most_half_step():
    rng = np.random.default_rng(7)
    x = (rng.standard_normal((400, 48)) * rng.uniform(0.1, 10, (400, 1))).astype(np.float32)
    codes, params = oracle.quantize_rows(x)
    deq = oracle.dequantize_rows(codes, params)
    err = np.abs(deq.astype(np.float64) - x)
    bound = params[:, 1:2].astype(np.float64) * 0.5 + 4 * np.spacing(np.abs(x)).astype(np.float64)
    assert np.all(err <= bound)


def test_signed_zero_extremes_are_positive_zero():
    x = np.array([[-0.0, 0.0, -0.0, 0.0], [0.0, -0.0, -0.0, -0.0], [-0.0] * 4, [-1.0, -0.0, -0.5, 0.0]], np.float32)
    codes, params = oracle.quantize_rows(x)
    assert not np.signbit(params[:3, 0]).any() and np.all(params[:3, 1] == 0)
    assert params[3, 1] == np.float32(1.0) / np.float32(255.0)


def test_constant_row():
    x = np.full((3, 8), 0.3, np.float32)
    x[1] = -2.0
    x[2] = 0.0
    codes, params = oracle.quantize_rows(x)
    assert np.all(codes == 0) and np.all(params[:, 1] == 0)
    deq = oracle.dequantize_rows(codes, params)
    assert np.all(np.abs(deq - x) <= np.spacing(np.abs(x) + np.float32(1e-38)))


def test_size_reduction_example():
    g = json.load(open(os.path.join(GOLDEN, "quant_size_example.json")))
    src = g["rows"] * g["dim"] * g["source_bytes_per_value"]
    q = g["rows"] * (g["dim"] * g["bits"] // 8 + g["row_values_kept"] * 4)
    assert 1 - q / src > g["reduction_over"]


def test_dequantize_matches_float64_formula():
    rng = np.random.default_rng(9)
    x = rng.standard_normal((64, 32)).astype(np.float32)
    codes, params = oracle.quantize_rows(x)
    # code * scale is exact in float64 (8 + 24 significant bits), and so is adding middle
    # here; one rounding to float32 is then the fused multiply-add's result
    ref = (codes.astype(np.float64) * params[:, 1:2].astype(np.float64) + params[:, 0:1].astype(np.float64))
    assert np.array_equal(oracle.dequantize_rows(codes, params), ref.astype(np.float32))


@pytest.mark.parametrize("combine,bf16", [("sum", True), ("mul", False)])
def test_gather_q8_vs_onehot(combine, bf16):
    wl = WORKLOADS["small"].with_(batch=128, combine=combine)
    inp = make_inputs(wl, with_weights=False, with_grad=False)
    B, F, D, Nd, V, m = 128, wl.num_cat, wl.emb_dim, wl.num_dense, wl.vocab, wl.table_rows
    qc, qp = oracle.quantize_rows(inp["q_tables"].float().numpy().reshape(F * m, D))
    rc, rp = oracle.quantize_rows(inp["r_tables"].float().numpy().reshape(F * m, D))
    ids = inp["ids"].numpy()
    x0, bad = oracle.gather_q8(B, F, D, Nd, V, m, m, combine, bf16, ids, None, qc, qp, rc, rp, inp["dense"])
    assert bad == 0
    deq = lambda c, p: (c.astype(np.float64) * p[:, 1:2] + p[:, 0:1]).astype(np.float32).reshape(F, m, D)
    qd, rd = deq(qc, qp), deq(rc, rp)
    for f in (0, 7, F - 1):
        q = qd[f][ids[:, f] // m]
        r = rd[f][ids[:, f] % m]
        e = (q * r) if combine == "mul" else (q + r)  # float32 elementwise, one rounding each
        if bf16:
            e = oracle.round_bf16(e)
        assert np.array_equal(x0[:, f * D:(f + 1) * D], e)
