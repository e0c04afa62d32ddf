"""Pins for the oracle's QR index (section 'Model Dictionary Compression').

The quotient/remainder split is Euclidean division by the remainder-table size
m: id = qi*m + ri with 0 <= ri < m. These tests check that defining property
exhaustively over every workload's vocabulary (so the map is a bijection onto
the first V (qi, ri) pairs, i.e. collision-free), the paper's worked sizing
example, and the uniqueness of combined embeddings the paper claims.
"""
import json
import os

import numpy as np
import pytest

import oracle
from paper_2402_06859_amd.synth import WORKLOADS

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("name", list(WORKLOADS))
def test_qr_bijection_exhaustive(name):
    wl = WORKLOADS[name]
    V, m = wl.vocab, wl.table_rows
    ids = np.arange(V, dtype=np.int64)
    qi, ri, bad = oracle.qr_index(ids, V, m)
    assert bad == 0
    # Euclidean division: reconstruction and remainder range
    assert np.array_equal(qi * m + ri, ids)
    assert ri.min() == 0 and ri.max() == min(m, V) - 1
    rq = oracle.quotient_rows(V, m)
    assert qi.min() == 0 and qi.max() == rq - 1
    # both tables of the workload have m rows: the quotient rows must fit
    assert rq <= m and m * m >= V


def test_qr_out_of_range_flagged():
    ids = np.array([-1, 0, 9_999, 10_000, -(2 ** 62), 2 ** 62], dtype=np.int64)
    qi, ri, bad = oracle.qr_index(ids, 10_000, 100)
    assert bad == 4
    assert list(qi) == [-1, 0, 99, -1, -1, -1] and list(ri) == [-1, 0, 99, -1, -1, -1]


def test_qr_paper_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "qr_worked_example.json")))
    V, m = g["vocab"], g["remainder_rows"]
    rq = oracle.quotient_rows(V, m)
    assert abs(rq - g["quotient_rows_about"]) / g["quotient_rows_about"] < 0.01
    assert abs(V / (rq + m) - g["compression_about"]) / g["compression_about"] < 0.01
    qi, ri, bad = oracle.qr_index(np.array([0, V - 1], dtype=np.int64), V, m)
    assert bad == 0 and qi[1] == rq - 1 and ri[1] == m - 1


def test_combined_embeddings_unique_tiny():
    """Every id of the tiny vocabulary gets a distinct combined embedding ('preserving
    embedding uniqueness across IDs'), for random tables, with both combines."""
    wl = WORKLOADS["tiny"]
    rng = np.random.default_rng(7)
    V, m, D = wl.vocab, wl.table_rows, wl.emb_dim
    rq = oracle.quotient_rows(V, m)
    qt = rng.standard_normal((1, rq, D)).astype(np.float32)
    rt = rng.standard_normal((1, m, D)).astype(np.float32)
    ids = np.arange(V, dtype=np.int64).reshape(V, 1)
    for combine in ("mul", "sum"):
        x0, bad = oracle.gather(V, 1, D, 0, V, rq, m, combine, False, ids, None, qt, rt, np.zeros((V, 0), np.float32))
        assert bad == 0
        assert len(np.unique(x0, axis=0)) == V
