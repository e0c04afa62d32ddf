"""Row-parallel runs of the CPU oracle for the GPU parity tests (test infrastructure).

The oracle's cross-stack forward and backward take about a second per row at the
large workload's size, so comparisons over whole 256-row tiles split the rows over
single-threaded worker processes. The inputs go to the workers as memory-mapped
.npy files (written once); each worker returns its rows' outputs and its rows' share
of the weight gradients, which the parent sums (the gradients are sums over rows).
Nothing here computes anything itself: every value comes from oracle/.
"""
import multiprocessing as mp
import os
from concurrent.futures import ProcessPoolExecutor
import shutil
import tempfile

import numpy as np

_S = {}


def _init(tmp: str):
    for name in ("W", "U", "b", "x0", "G"):
        path = os.path.join(tmp, name + ".npy")
        if os.path.exists(path):
            _S[name] = np.load(path, mmap_mode="r")


def _forward(task):
    lo, hi, alpha, beta, tau, parallel = task
    import oracle
    W, U, b = list(_S["W"]), list(_S["U"]), list(_S["b"])
    return lo, oracle.forward(np.asarray(_S["x0"][lo:hi]), W, U, b, alpha, beta, tau, parallel=parallel)


def _backward(task):
    lo, hi, alpha, beta, tau, parallel = task
    import oracle
    W, U, b = list(_S["W"]), list(_S["U"]), list(_S["b"])
    gx0, gW, gU, gb = oracle.backward(np.asarray(_S["x0"][lo:hi]), W, U, b, np.asarray(_S["G"][lo:hi]), alpha,
                                      beta, tau, parallel=parallel)
    # partial weight gradients as float32 (a float64 sum over this chunk's rows, rounded once)
    return lo, gx0, gW.astype(np.float32), gU.astype(np.float32), gb


def default_workers(weight_bytes: int) -> int:
    """At most 16 processes (the host CPU share of one GPU), fewer when memory is short: each
    worker holds float64 copies of the weights and of their gradients."""
    n = min(16, os.cpu_count() or 1)
    try:
        with open("/proc/meminfo") as fh:
            avail = next(int(l.split()[1]) * 1024 for l in fh if l.startswith("MemAvailable:"))
        n = min(n, max(1, int(0.5 * avail // (6 * weight_bytes + (1 << 30)))))
    except (OSError, StopIteration):
        pass
    return max(1, n)


def dcn_oracle(x0, W, U, b, G, alpha, beta, tau, parallel=False, backward=True, workers=None):
    """Oracle forward x_L of every row of x0 [R, d] and, with backward, the gradients for
    upstream gradient G [R, d]: (xL, gx0, gW [L, n r, d], gU [L, d, hr], gb [L, d]), float64
    (weight gradients summed over the rows in float64 from float32 chunk partials)."""
    x0 = np.ascontiguousarray(x0, np.float32)
    R = x0.shape[0]
    Ws = np.stack([np.asarray(w, np.float32) for w in W])
    Us = np.stack([np.asarray(u, np.float32) for u in U])
    bs = np.stack([np.asarray(v, np.float32) for v in b])
    n = workers or default_workers(8 * (Ws.size + Us.size))
    bounds = np.linspace(0, R, min(R, 2 * n) + 1).astype(int)
    tasks = [(int(lo), int(hi), alpha, beta, tau, parallel) for lo, hi in zip(bounds[:-1], bounds[1:]) if hi > lo]
    tmp = tempfile.mkdtemp(prefix="orcpool_")
    try:
        np.save(os.path.join(tmp, "W.npy"), Ws)
        np.save(os.path.join(tmp, "U.npy"), Us)
        np.save(os.path.join(tmp, "b.npy"), bs)
        np.save(os.path.join(tmp, "x0.npy"), x0)
        if backward:
            np.save(os.path.join(tmp, "G.npy"), np.ascontiguousarray(G, np.float32))
        d = x0.shape[1]
        xL = np.empty((R, d))
        out = None
        # (a worker that dies raises BrokenProcessPool here instead of being replaced)
        with ProcessPoolExecutor(n, mp_context=mp.get_context("spawn"), initializer=_init, initargs=(tmp,)) as pool:
            for lo, y in pool.map(_forward, tasks):
                xL[lo:lo + y.shape[0]] = y
            if backward:
                gx0 = np.empty((R, d))
                gW = np.zeros(Ws.shape)
                gU = np.zeros(Us.shape)
                gb = np.zeros(bs.shape)
                for lo, g0, pw, pu, pb in pool.map(_backward, tasks):
                    gx0[lo:lo + g0.shape[0]] = g0
                    gW += pw
                    gU += pu
                    gb += pb
                out = (gx0, gW, gU, gb)
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    return (xL,) + out if backward else xL
