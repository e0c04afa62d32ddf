"""Workload registry and seeded synthetic inputs for the Residual-DCN + QR-embedding path.

This module only describes and draws inputs: shapes, value distributions and
seeds. It contains none of the method's arithmetic (no hashing, combining,
cross layers or gradients), so the CPU oracle and the HIP path can both be fed
from it without sharing any computation.

Workloads (LiRank, KDD'24): the paper's data is LinkedIn production traffic,
which is not available; these synthetic batches stand in for it with the shapes
of a ranking model input -- categorical ids with a heavy-tailed (Zipf)
frequency, per-feature quotient/remainder tables (Model Dictionary Compression
section), dense features concatenated after the embeddings (appendix, Feed
Ranking Sparse ID features) and a stack of Residual DCN layers (Residual DCN
section).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np

SEED_BASE = 240206859


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    index: int            # seed offset
    batch: int            # B
    num_cat: int          # F categorical features
    vocab: int            # V ids per feature
    table_rows: int       # m: rows of every quotient and remainder table
    emb_dim: int          # D
    num_dense: int        # Nd
    num_layers: int       # L
    rank: int             # r
    attention: bool       # attention term + skip connection on (alpha, beta) = (1, 1)
    dtype: str            # "f32" or "bf16" storage
    combine: str          # "mul" or "sum"
    zipf_s: float
    multi_hot: bool = False
    bag_mean: float = 20.0
    bag_min: int = 1
    bag_max: int = 100
    dense_zero_frac: float = 0.0
    temperature: float = 1.0
    skip_beta: float = 1.0
    act_mode: str = "storage"        # x_l and h: storage type, "hilo" bf16 pairs or "f16" (deep attention stacks)
    parallel: bool = False           # plain + attention low-rank cross nets with their own weights
    hashed: bool = False             # Murmur front-end: two QR table pairs per feature, rows*rows >= 2^32
    hash_seed: int = 0

    @property
    def d(self) -> int:
        return self.num_cat * self.emb_dim + self.num_dense

    @property
    def table_pairs(self) -> int:
        return 2 if self.hashed else 1

    @property
    def quotient_rows_used(self) -> int:
        # number of quotient-table rows that ids in [0, V) can reach
        return -(-self.vocab // self.table_rows)

    @property
    def alpha(self) -> float:
        return 1.0 if self.attention else 0.0

    @property
    def beta(self) -> float:
        return self.skip_beta

    @property
    def n_proj(self) -> int:
        return (4 if self.parallel else 3) if self.attention else 1

    @property
    def h_width(self) -> int:
        """Width of the up projection's input (2r with parallel branches)."""
        return 2 * self.rank if (self.parallel and self.attention) else self.rank

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", 0, 512, 8, 10_000, 100, 16, 32, 2, 32, False, "f32", "mul", 1.1),
    "small": Workload("small", 1, 4096, 50, 1_000_000, 1000, 32, 256, 3, 256, True, "bf16", "sum", 1.1),
    "feed": Workload("feed", 2, 16384, 120, 5_000_000, 2237, 32, 512, 4, 512, False, "bf16", "sum", 1.05,
                     dense_zero_frac=0.05),
    "multihot": Workload("multihot", 3, 8192, 64, 10_000_000, 3163, 64, 256, 3, 512, False, "bf16", "sum", 1.1,
                         multi_hot=True),
    "large": Workload("large", 4, 32768, 200, 20_000_000, 4473, 48, 1024, 6, 1024, True, "bf16", "sum", 1.1,
                      act_mode="f16"),
}


def _streams(wl: Workload, seed: Optional[int]) -> Dict[str, np.random.Generator]:
    base = SEED_BASE + wl.index if seed is None else seed
    names = ["ids", "lens", "dense", "tables", "weights", "grad", "scatter"]
    ss = np.random.SeedSequence(base).spawn(len(names))
    return {n: np.random.Generator(np.random.PCG64(s)) for n, s in zip(names, ss)}


def zipf_ranks(rng: np.random.Generator, s: float, vmax: int, n: int) -> np.ndarray:
    """n draws of a Zipf(s) rank in [1, vmax] (truncated by rejection)."""
    out = np.empty(n, dtype=np.int64)
    filled = 0
    while filled < n:
        want = int((n - filled) * 2.2) + 64
        k = rng.zipf(s, size=want)
        k = k[k <= vmax]
        take = min(len(k), n - filled)
        out[filled:filled + take] = k[:take]
        filled += take
    return out


def scatter_params(rng: np.random.Generator, vocab: int, num_cat: int):
    """Per-feature (a_f, c_f) with gcd(a_f, V) = 1: rank k -> id (a_f*(k-1)+c_f) mod V is a bijection."""
    a = np.empty(num_cat, dtype=np.int64)
    c = np.empty(num_cat, dtype=np.int64)
    for f in range(num_cat):
        while True:
            cand = int(rng.integers(vocab // 3 + 1, vocab)) | 1
            if math.gcd(cand, vocab) == 1:
                break
        a[f] = cand
        c[f] = int(rng.integers(0, vocab))
    return a, c


def ranks_to_ids(ranks: np.ndarray, feat: np.ndarray, vocab: int, a: np.ndarray, c: np.ndarray,
                 mode: str) -> np.ndarray:
    if mode == "rank":
        return ranks - 1
    # (a*(k-1) + c) mod V without int64 overflow: a < V <= 2^31, k-1 < V
    k = (ranks - 1).astype(object) if vocab > (1 << 31) else (ranks - 1)
    ids = (a[feat].astype(np.uint64) * k.astype(np.uint64) + c[feat].astype(np.uint64)) % np.uint64(vocab)
    return ids.astype(np.int64)


def to_storage(x: np.ndarray, dtype: str):
    """float32 numpy -> torch CPU tensor in the storage dtype (bf16 rounding done by torch, RNE)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def storage_values(t) -> np.ndarray:
    """torch CPU tensor (bf16 or f32) -> float32 numpy holding exactly the stored values."""
    return t.float().numpy()


def make_inputs(wl: Workload, seed: Optional[int] = None, id_mode: str = "scatter",
                batch: Optional[int] = None, with_grad: bool = True,
                with_weights: bool = True, bias_std: float = 0.0) -> dict:
    """Draw one synthetic batch for workload `wl`.

    Returns torch CPU tensors in the storage dtype (tables, dense, weights, grad_out),
    int64 ids (and int64 CSR offsets for multi-hot), plus metadata. Weight layout per
    layer l: w_down[l] is [n*r, d] with row blocks (value, query, key) -- the value
    block alone when the attention term is off -- u[l] is [d, r], bias[l] is [d].
    """
    import torch
    B = wl.batch if batch is None else batch
    st = _streams(wl, seed)
    F, V, m, D = wl.num_cat, wl.vocab, wl.table_rows, wl.emb_dim
    out: dict = {"workload": wl, "batch": B}

    a, c = scatter_params(st["scatter"], V, F)
    if wl.multi_hot:
        lens = st["lens"].poisson(wl.bag_mean, size=(B, F)).clip(wl.bag_min, wl.bag_max).astype(np.int64)
        offsets = np.zeros(B * F + 1, dtype=np.int64)
        np.cumsum(lens.reshape(-1), out=offsets[1:])
        nnz = int(offsets[-1])
        feat = np.repeat(np.tile(np.arange(F, dtype=np.int64), B), lens.reshape(-1))
        ranks = zipf_ranks(st["ids"], wl.zipf_s, V, nnz)
        ids = ranks_to_ids(ranks, feat, V, a, c, id_mode)
        out["ids"] = torch.from_numpy(ids)
        out["offsets"] = torch.from_numpy(offsets)
    else:
        feat = np.tile(np.arange(F, dtype=np.int64), B)
        ranks = zipf_ranks(st["ids"], wl.zipf_s, V, B * F)
        ids = ranks_to_ids(ranks, feat, V, a, c, id_mode)
        out["ids"] = torch.from_numpy(ids.reshape(B, F))
        out["offsets"] = None

    # tables: N(0, sigma^2); sigma = 1 for the multiplicative combine, 1/sqrt(2) for the additive one
    sigma = 1.0 if wl.combine == "mul" else 1.0 / math.sqrt(2.0)
    tg = st["tables"]
    shape = (F, 2, m, D) if wl.hashed else (F, m, D)  # hashed: one (Q, R) pair per hash half
    out["q_tables"] = to_storage(tg.standard_normal(shape, dtype=np.float32) * sigma, wl.dtype)
    out["r_tables"] = to_storage(tg.standard_normal(shape, dtype=np.float32) * sigma, wl.dtype)

    dense = st["dense"].standard_normal((B, wl.num_dense), dtype=np.float32)
    if wl.dense_zero_frac > 0:
        dense[st["dense"].random((B, wl.num_dense)) < wl.dense_zero_frac] = 0.0
    out["dense"] = to_storage(dense, wl.dtype)

    if with_weights:
        out.update(make_weights(wl, st["weights"], bias_std))
    if with_grad:
        out["grad_out"] = to_storage(st["grad"].standard_normal((B, wl.d), dtype=np.float32), wl.dtype)
    return out


def make_weights(wl: Workload, rng: np.random.Generator, bias_std: float = 0.0) -> dict:
    """Xavier-normal projections (std sqrt(2/(d+r))), bias N(0, bias_std^2) (0 by default).
    With parallel branches w_down stacks (V1, V2, Q, K) and u is [U1 | U2]."""
    d, r, n = wl.d, wl.rank, wl.n_proj
    std = math.sqrt(2.0 / (d + r))
    w_down: List = []
    u: List = []
    bias: List = []
    for _ in range(wl.num_layers):
        w_down.append(to_storage(rng.standard_normal((n * r, d), dtype=np.float32) * std, wl.dtype))
        u.append(to_storage(rng.standard_normal((d, wl.h_width), dtype=np.float32) * std, wl.dtype))
        b = rng.standard_normal(d, dtype=np.float32) * bias_std if bias_std > 0 else np.zeros(d, np.float32)
        bias.append(to_storage(b, wl.dtype))
    return {"w_down": w_down, "u": u, "bias": bias}


def grad_x0_like(wl: Workload, B: int, seed: int):
    """Seeded fp32 upstream gradient for the x0 rows (input of the embedding backward)."""
    import torch
    rng = np.random.Generator(np.random.PCG64(seed))
    return torch.from_numpy(rng.standard_normal((B, wl.d), dtype=np.float32))


# ---------------------------------------------------------------------------
# Head after the cross stack (section "Dense Gating and Large MLP", section
# "Isotonic Calibration Layer"): gated wide ReLU layers, a logit, calibration.
# ---------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class HeadSpec:
    name: str
    hidden: tuple            # logical widths (the Feed "Large MLP" is 4 x 3500)
    gated: bool = True
    buckets: int = 32        # K calibration buckets over [lo, lo + K*step]
    lo: float = -4.0
    step: float = 0.25
    gate_bias: float = 1.0   # initial gate logit offset (gates start mostly open)
    e_std: float = 0.1       # per-sample calibration embedding values
    label_rate: float = 0.1  # positive rate of the synthetic binary labels

    @property
    def widths(self) -> tuple:
        """Stored widths: each logical width rounded up to a multiple of 8; the extra
        units have zero weights and biases, so the model is exactly the logical one."""
        return tuple(-(-n // 8) * 8 for n in self.hidden)


HEADS: Dict[str, HeadSpec] = {
    "lmlp": HeadSpec("lmlp", (3500, 3500, 3500, 3500)),
    "small": HeadSpec("small", (256, 128)),
}


def make_head_inputs(wl: Workload, head: HeadSpec, batch: Optional[int] = None, seed: Optional[int] = None,
                     with_x: bool = True, bias_std: float = 0.05) -> dict:
    """Seeded head parameters and per-sample inputs (torch CPU tensors).

    W[l] [n_l, n_{l-1}] bf16 He-normal (std sqrt(2/n_{l-1}) over the logical fan-in),
    b[l] N(0, bias_std^2), gate weights G[l] [n_{l-1}] N(0, 1/n_{l-1}) and gate bias
    c[l] [1] = gate_bias, w_out N(0, 1/n_L), b_out 0, cal_w U(0.5, 1.5) float, cal_b 0;
    e [B, K] N(0, e_std^2) float, labels Bernoulli(label_rate) float, g_cal [B] N(0, 1)
    float (an upstream gradient for tests); x [B, d] bf16 N(0, 1) when with_x. Units
    beyond a logical width have zero weights, biases, gate and output weights."""
    B = wl.batch if batch is None else batch
    base = SEED_BASE + 1000 + wl.index if seed is None else seed
    ss = np.random.SeedSequence(base).spawn(4)
    rw, rc, rx, rg = (np.random.Generator(np.random.PCG64(s)) for s in ss)
    logical = (wl.d,) + tuple(head.hidden)
    stored = (wl.d,) + head.widths
    W, b, G, c = [], [], [], []
    for l in range(len(head.hidden)):
        nin, nout = stored[l], stored[l + 1]
        w = np.zeros((nout, nin), np.float32)
        w[:logical[l + 1], :logical[l]] = rw.standard_normal((logical[l + 1], logical[l]), dtype=np.float32) * \
            math.sqrt(2.0 / logical[l])
        bv = np.zeros(nout, np.float32)
        bv[:logical[l + 1]] = rw.standard_normal(logical[l + 1], dtype=np.float32) * bias_std
        g = np.zeros(nin, np.float32)
        g[:logical[l]] = rw.standard_normal(logical[l], dtype=np.float32) / math.sqrt(logical[l])
        W.append(to_storage(w, "bf16"))
        b.append(to_storage(bv, "bf16"))
        G.append(to_storage(g, "bf16"))
        c.append(to_storage(np.array([head.gate_bias], np.float32), "bf16"))
    wo = np.zeros(stored[-1], np.float32)
    wo[:logical[-1]] = rw.standard_normal(logical[-1], dtype=np.float32) / math.sqrt(logical[-1])
    K = head.buckets
    import torch
    out = {"W": W, "b": b, "w_out": to_storage(wo, "bf16"), "b_out": to_storage(np.zeros(1, np.float32), "bf16"),
           "cal_w": torch.from_numpy(rc.uniform(0.5, 1.5, K).astype(np.float32)),
           "cal_b": torch.zeros(1, dtype=torch.float32),
           "e": torch.from_numpy(rc.standard_normal((B, K), dtype=np.float32) * head.e_std),
           "labels": torch.from_numpy((rc.random(B) < head.label_rate).astype(np.float32)),
           "g_cal": torch.from_numpy(rg.standard_normal(B, dtype=np.float32))}
    if head.gated:
        out["G"], out["c"] = G, c
    if with_x:
        out["x"] = to_storage(rx.standard_normal((B, wl.d), dtype=np.float32), "bf16")
    return out
