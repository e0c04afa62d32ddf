"""Shared helpers of the GPU parity tests (test infrastructure)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2402_06859_amd.synth import Workload


def need_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need an MI355X; torch.cuda.is_available() is False")


def relerr(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / (den if den > 0 else 1.0))


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy()


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().view(torch.int16).numpy()


def oracle_x0(wl: Workload, inp: dict) -> np.ndarray:
    x0, bad = oracle.gather(inp["batch"], wl.num_cat, wl.emb_dim, wl.num_dense, wl.vocab, wl.table_rows,
                            wl.table_rows, wl.combine, wl.dtype == "bf16", inp["ids"], inp["offsets"],
                            inp["q_tables"], inp["r_tables"], inp["dense"])
    assert bad == 0
    return x0


def sample_rows(B: int, k: int) -> np.ndarray:
    """k distinct rows spread over [0, B), always including the first and the last."""
    if k >= B:
        return np.arange(B)
    rows = np.unique(np.concatenate([[0, B - 1], np.linspace(0, B - 1, k).astype(np.int64),
                                     np.random.default_rng(B).choice(B, k // 2, replace=False)]))
    return rows


FWD_TOL = {"f32": 1e-5, "bf16": 2e-2}
GRAD_TOL = 5e-2
