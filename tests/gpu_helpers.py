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


# A tensor passes when its normwise relative error is within tol (the stated bar),
# every row's and column's error within block * tol of the larger of its own norm and
# the tensor's typical (RMS) row or column norm, and every element's error within
# elem * tol of the larger of its own size and the tensor's RMS. A wrong row, column or
# element of ordinary size is off by about 1 on that scale (2 with a wrong sign); rows,
# columns and elements much smaller than typical are judged on the typical scale, where
# the rounding errors of the other terms set their absolute error. Forward outputs use
# (block, elem) = (3, 10). Gradients use (5, 20): the query and key weight gradients of
# a sharp softmax are sums whose terms are very sensitive to rounding (measured worst:
# a row at 0.21 and an element at 0.84 of their scale, with tau = 0.25 and on the large
# workload's near one-hot last layers, where the normwise errors were 0.034 and 0.015).
FWD_GATES = (3.0, 10.0)
GRAD_GATES = (5.0, 20.0)


def error_stats(got, ref) -> dict:
    """Normwise relative error, and the worst row, column and element errors on the scales
    described above (rows and columns of 2-D tensors only)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    diff = got - ref
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    scale = np.maximum(np.abs(ref), rms)
    out = {"norm": relerr(got, ref)}
    out["elem"] = float(np.max(np.abs(diff) / scale)) if rms > 0 else float(np.max(np.abs(diff), initial=0.0))
    if ref.ndim == 2 and rms > 0:
        for axis, key in ((1, "row"), (0, "col")):
            num = np.linalg.norm(diff, axis=axis)
            den = np.linalg.norm(ref, axis=axis)
            typical = float(np.sqrt(np.mean(den * den)))
            out[key] = float(np.max(num / np.maximum(den, typical)))
    return out


def check_tensor(name: str, got, ref, tol: float, errs: dict, gates=FWD_GATES):
    """Record error_stats(got, ref) under `name` in errs; return the list of failed gates
    (gates = (block, elem) factors, see above)."""
    block, elem = gates
    e = error_stats(got, ref)
    errs[name] = e
    bad = []
    if not e["norm"] <= tol:
        bad.append("%s norm %.3g > %.3g" % (name, e["norm"], tol))
    for key in ("row", "col"):
        if key in e and not e[key] <= block * tol:
            bad.append("%s %s %.3g > %.3g" % (name, key, e[key], block * tol))
    if not e["elem"] <= elem * tol:
        bad.append("%s elem %.3g > %.3g" % (name, e["elem"], elem * tol))
    return bad


def tile_rows(B: int, tile: int = 256) -> np.ndarray:
    """Whole contiguous row tiles: [0, tile), one tile in the middle, and the last (possibly
    partial) tile; all rows when B is at most three tiles."""
    if B <= 3 * tile:
        return np.arange(B)
    mid = (B // 2) // tile * tile
    last = (B - 1) // tile * tile
    return np.unique(np.concatenate([np.arange(0, tile), np.arange(mid, mid + tile), np.arange(last, B)]))


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
