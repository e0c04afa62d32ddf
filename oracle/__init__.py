"""CPU oracle for the Residual-DCN + QR-embedding path -- TEST INFRASTRUCTURE ONLY.

Plain C loops (oracle.c) behind ctypes. Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import this package; the product library and
its Python binding never do. See oracle.c for the paper passages each
function follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

COMBINE = {"mul": 0, "sum": 1}


def build(force: bool = True) -> str:
    """Compile oracle.c with gcc (no fused multiply-add, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
                               "-shared", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        L = ctypes.CDLL(_LIB)
        i64, dbl, vp = ctypes.c_int64, ctypes.c_double, ctypes.c_void_p
        L.orc_qr_quotient_rows.argtypes = [i64, i64]
        L.orc_qr_quotient_rows.restype = i64
        L.orc_qr_index.argtypes = [vp, i64, i64, i64, vp, vp]
        L.orc_qr_index.restype = i64
        L.orc_round_bf16_array.argtypes = [vp, vp, i64]
        L.orc_round_bf16_array.restype = None
        L.orc_gather.argtypes = [i64, i64, i64, i64, i64, i64, i64, ctypes.c_int, ctypes.c_int,
                                 vp, vp, vp, vp, vp, vp]
        L.orc_gather.restype = i64
        L.orc_attention.argtypes = [i64, dbl, dbl, dbl, vp, vp, vp, vp, vp, vp]
        L.orc_attention.restype = None
        L.orc_forward.argtypes = [i64, i64, i64, i64, dbl, dbl, dbl, ctypes.c_int, vp, vp, vp, vp, vp]
        L.orc_forward.restype = ctypes.c_int
        L.orc_backward.argtypes = [i64, i64, i64, i64, dbl, dbl, dbl, ctypes.c_int, vp, vp, vp, vp, vp, vp, vp, vp,
                                   vp]
        L.orc_backward.restype = ctypes.c_int
        L.orc_embed_backward.argtypes = [i64, i64, i64, i64, i64, i64, i64, ctypes.c_int, vp, vp, vp, vp, vp,
                                         vp, vp]
        L.orc_embed_backward.restype = i64
        L.orc_quantize_rows.argtypes = [i64, i64, vp, vp, vp]
        L.orc_quantize_rows.restype = ctypes.c_int
        L.orc_dequantize_rows.argtypes = [i64, i64, vp, vp, vp]
        L.orc_dequantize_rows.restype = ctypes.c_int
        L.orc_gather_q8.argtypes = [i64, i64, i64, i64, i64, i64, i64, ctypes.c_int, ctypes.c_int, vp, vp, vp, vp,
                                    vp, vp, vp, vp]
        L.orc_gather_q8.restype = i64
        u64 = ctypes.c_uint64
        L.orc_murmur64a.argtypes = [vp, i64, u64]
        L.orc_murmur64a.restype = u64
        L.orc_hash_ids.argtypes = [vp, i64, u64, vp]
        L.orc_hash_ids.restype = None
        L.orc_gather_hashed.argtypes = [i64, i64, i64, i64, i64, i64, ctypes.c_int, ctypes.c_int, u64, vp, vp, vp, vp,
                                        vp, vp]
        L.orc_gather_hashed.restype = i64
        L.orc_embed_backward_hashed.argtypes = [i64, i64, i64, i64, i64, i64, ctypes.c_int, u64, vp, vp, vp, vp, vp,
                                                vp, vp]
        L.orc_embed_backward_hashed.restype = i64
        _lib = L
    return _lib


def _c(a: np.ndarray, dtype) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def _np(x, dtype):
    if x is None:
        return None
    if hasattr(x, "numpy"):  # torch CPU tensor
        x = x.float().numpy() if dtype in (np.float32, np.float64) else x.numpy()
    return _c(x, dtype)


def quotient_rows(vocab: int, m: int) -> int:
    return int(lib().orc_qr_quotient_rows(vocab, m))


def qr_index(ids, vocab: int, m: int):
    ids = _np(ids, np.int64).reshape(-1)
    qi = np.empty_like(ids)
    ri = np.empty_like(ids)
    bad = lib().orc_qr_index(_p(ids), ids.size, vocab, m, _p(qi), _p(ri))
    return qi, ri, int(bad)


def round_bf16(x) -> np.ndarray:
    x = _np(x, np.float32)
    y = np.empty_like(x)
    lib().orc_round_bf16_array(_p(x), _p(y), x.size)
    return y


def round_f16(x) -> np.ndarray:
    """x (as float32) rounded to the nearest IEEE binary16 value, ties to even,
    |x| >= 65520 to infinity, returned as float32: the rounding of an activation
    kept in f16. numpy's float16 cast is the rounding step."""
    return np.asarray(x, np.float32).astype(np.float16).astype(np.float32)


def gather(B: int, F: int, D: int, Nd: int, vocab: int, rows_q: int, m: int, combine: str, bf16: bool,
           ids, offsets, q_tables, r_tables, dense):
    """x0 [B, F*D+Nd] float32 (bf16-rounded values when bf16) and the out-of-range id count."""
    ids = _np(ids, np.int64)
    offsets = _np(offsets, np.int64)
    qt = _np(q_tables, np.float32)
    rt = _np(r_tables, np.float32)
    dn = _np(dense, np.float32)
    x0 = np.empty((B, F * D + Nd), np.float32)
    bad = lib().orc_gather(B, F, D, Nd, vocab, rows_q, m, COMBINE[combine], int(bf16), _p(ids), _p(offsets),
                           _p(qt), _p(rt), _p(dn), _p(x0))
    if bad < 0:
        raise ValueError("orc_gather: bad arguments")
    return x0, int(bad)


def attention(q, k, v, alpha: float, beta: float, tau: float):
    """One sample: returns (A [r, r], o [r], h [r]) in float64."""
    q, k, v = (_c(np.asarray(a), np.float64) for a in (q, k, v))
    r = q.size
    A = np.empty((r, r))
    o = np.empty(r)
    h = np.empty(r)
    lib().orc_attention(r, alpha, beta, tau, _p(q), _p(k), _p(v), _p(A), _p(o), _p(h))
    return A, o, h


def _stack(ws: Sequence, dtype=np.float64) -> np.ndarray:
    return _c(np.stack([_np(w, np.float64) for w in ws]), dtype)


def _rank(U, parallel: bool) -> int:
    return U.shape[2] // (2 if parallel else 1)


def forward(x0, w_down: Sequence, u: Sequence, bias: Sequence, alpha: float, beta: float, tau: float = 1.0,
            parallel: bool = False):
    """x_L [B, d] in float64 from storage values (x0, weights as float arrays / torch tensors).
    parallel: a plain and an attention low-rank cross net with their own weights per layer
    (w_down [4r, d] = V1, V2, Q, K; u [d, 2r] = [U1 | U2])."""
    x0 = _np(x0, np.float64)
    B, d = x0.shape
    L = len(w_down)
    W, U, b = _stack(w_down), _stack(u), _stack(bias)
    r = _rank(U, parallel)
    out = np.empty((B, d))
    rc = lib().orc_forward(B, d, r, L, alpha, beta, tau, int(parallel), _p(x0), _p(W), _p(U), _p(b), _p(out))
    if rc != 0:
        raise ValueError("orc_forward: bad arguments")
    return out


def backward(x0, w_down: Sequence, u: Sequence, bias: Sequence, grad_out, alpha: float, beta: float,
             tau: float = 1.0, parallel: bool = False):
    """(grad_x0 [B, d], g_w_down [L, n*r, d], g_u [L, d, hr], g_bias [L, d]) in float64."""
    x0 = _np(x0, np.float64)
    G = _np(grad_out, np.float64)
    B, d = x0.shape
    L = len(w_down)
    W, U, b = _stack(w_down), _stack(u), _stack(bias)
    r = _rank(U, parallel)
    gx0 = np.empty((B, d))
    gW = np.empty_like(W)
    gU = np.empty_like(U)
    gb = np.empty_like(b)
    rc = lib().orc_backward(B, d, r, L, alpha, beta, tau, int(parallel), _p(x0), _p(W), _p(U), _p(b), _p(G),
                            _p(gx0), _p(gW),
                            _p(gU), _p(gb))
    if rc != 0:
        raise ValueError("orc_backward: bad arguments")
    return gx0, gW, gU, gb


def embed_backward(B: int, F: int, D: int, Nd: int, vocab: int, rows_q: int, m: int, combine: str, ids, offsets,
                   q_tables, r_tables, grad_x0, grad_q=None, grad_r=None):
    """Table gradients (float64, accumulated into grad_q / grad_r when given) and the bad-id count."""
    ids = _np(ids, np.int64)
    offsets = _np(offsets, np.int64)
    qt = _np(q_tables, np.float32)
    rt = _np(r_tables, np.float32)
    g = _np(grad_x0, np.float64)
    gq = np.zeros((F, rows_q, D)) if grad_q is None else _c(grad_q, np.float64)
    gr = np.zeros((F, m, D)) if grad_r is None else _c(grad_r, np.float64)
    bad = lib().orc_embed_backward(B, F, D, Nd, vocab, rows_q, m, COMBINE[combine], _p(ids), _p(offsets), _p(qt),
                                   _p(rt), _p(g), _p(gq), _p(gr))
    if bad < 0:
        raise ValueError("orc_embed_backward: bad arguments")
    return gq, gr, int(bad)


def quantize_rows(x):
    """Middle-max 8-bit row-wise quantization of x [rows, D] (float32 values):
    (codes int8 [rows, D], params float32 [rows, 2] = (middle, scale))."""
    x = _np(x, np.float32)
    rows, D = x.shape
    codes = np.empty((rows, D), np.int8)
    params = np.empty((rows, 2), np.float32)
    if lib().orc_quantize_rows(rows, D, _p(x), _p(codes), _p(params)) != 0:
        raise ValueError("orc_quantize_rows: bad arguments")
    return codes, params


def dequantize_rows(codes, params):
    codes = _c(codes, np.int8)
    params = _c(params, np.float32)
    rows, D = codes.shape
    x = np.empty((rows, D), np.float32)
    if lib().orc_dequantize_rows(rows, D, _p(codes), _p(params), _p(x)) != 0:
        raise ValueError("orc_dequantize_rows: bad arguments")
    return x


def gather_q8(B: int, F: int, D: int, Nd: int, vocab: int, rows_q: int, m: int, combine: str, bf16: bool,
              ids, offsets, q_codes, q_params, r_codes, r_params, dense):
    """Serving gather from quantized tables (codes [F*rows, D] int8, params [F*rows, 2]):
    x0 [B, F*D+Nd] float32 and the out-of-range id count."""
    ids = _np(ids, np.int64)
    offsets = _np(offsets, np.int64)
    qc, rc = _c(q_codes, np.int8), _c(r_codes, np.int8)
    qp, rp = _c(q_params, np.float32), _c(r_params, np.float32)
    dn = _np(dense, np.float32)
    x0 = np.empty((B, F * D + Nd), np.float32)
    bad = lib().orc_gather_q8(B, F, D, Nd, vocab, rows_q, m, COMBINE[combine], int(bf16), _p(ids), _p(offsets),
                              _p(qc), _p(qp), _p(rc), _p(rp), _p(dn), _p(x0))
    if bad < 0:
        raise ValueError("orc_gather_q8: bad arguments")
    return x0, int(bad)


def murmur64a(data: bytes, seed: int = 0) -> int:
    """MurmurHash64A of a byte string."""
    buf = ctypes.create_string_buffer(bytes(data), max(len(data), 1))
    return int(lib().orc_murmur64a(buf, len(data), seed))


def hash_ids(ids, seed: int = 0) -> np.ndarray:
    """uint64 MurmurHash64A of each id's 8 little-endian bytes."""
    ids = _np(ids, np.int64).reshape(-1)
    out = np.empty(ids.size, np.uint64)
    lib().orc_hash_ids(_p(ids), ids.size, seed, _p(out))
    return out


def gather_hashed(B: int, F: int, D: int, Nd: int, rows_q: int, m: int, combine: str, bf16: bool, seed: int,
                  ids, offsets, q_tables, r_tables, dense):
    """x0 [B, F*D+Nd] float32 of the hashed front-end (tables [F, 2, rows, D])."""
    ids = _np(ids, np.int64)
    offsets = _np(offsets, np.int64)
    qt = _np(q_tables, np.float32)
    rt = _np(r_tables, np.float32)
    dn = _np(dense, np.float32)
    x0 = np.empty((B, F * D + Nd), np.float32)
    rc = lib().orc_gather_hashed(B, F, D, Nd, rows_q, m, COMBINE[combine], int(bf16), seed, _p(ids), _p(offsets),
                                 _p(qt), _p(rt), _p(dn), _p(x0))
    if rc < 0:
        raise ValueError("orc_gather_hashed: bad arguments")
    return x0


def embed_backward_hashed(B: int, F: int, D: int, Nd: int, rows_q: int, m: int, combine: str, seed: int, ids,
                          offsets, q_tables, r_tables, grad_x0):
    """Table gradients (float64 [F, 2, rows, D]) of the hashed front-end."""
    ids = _np(ids, np.int64)
    offsets = _np(offsets, np.int64)
    qt = _np(q_tables, np.float32)
    rt = _np(r_tables, np.float32)
    g = _np(grad_x0, np.float64)
    gq = np.zeros((F, 2, rows_q, D))
    gr = np.zeros((F, 2, m, D))
    rc = lib().orc_embed_backward_hashed(B, F, D, Nd, rows_q, m, COMBINE[combine], seed, _p(ids), _p(offsets),
                                         _p(qt), _p(rt), _p(g), _p(gq), _p(gr))
    if rc < 0:
        raise ValueError("orc_embed_backward_hashed: bad arguments")
    return gq, gr
