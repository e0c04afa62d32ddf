"""Python binding of librdcn (include/rdcn.h): argument marshalling only.

Every computation runs in the library's HIP kernels; torch is used for device
memory and the current stream. If the shared library is missing it is built
with hipcc; if it cannot be loaded, an error is raised (there is no fallback).
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librdcn.so")
MAX_LAYERS = 16

(RDCN_OK, RDCN_ERR_ARG, RDCN_ERR_SHAPE, RDCN_ERR_INDEX, RDCN_ERR_UNSUPPORTED, RDCN_ERR_WORKSPACE, RDCN_ERR_HIP,
 RDCN_ERR_RANGE) = range(8)
F32, BF16 = 0, 1
I32, I64 = 0, 1
COMBINE_MUL, COMBINE_SUM = 0, 1
ACT_MODES = {"storage": 0, "hilo": 1, "f16": 2}   # rdcn_act_mode

EXPORTS = ["rdcn_create", "rdcn_destroy", "rdcn_dim", "rdcn_workspace_bytes", "qr_embed_gather",
           "qr_embed_backward_workspace", "qr_embed_backward", "rdcn_forward", "rdcn_backward",
           "rdcn_check_device_errors", "rdcn_status_string", "rdcn_profile_start", "rdcn_profile_stop",
           "qr_quantize_tables", "qr_embed_gather_q8", "rdcn_head_configure", "rdcn_head_workspace_bytes",
           "rdcn_head_forward", "rdcn_head_logloss", "rdcn_head_backward", "rdcn_set_side_stream",
           "qr_embed_backward_static"]
EMBED_STATIC_SCRATCH_BYTES = 64 << 20

KERNELS = ["gather", "fwd_down_gemm", "fwd_attention", "fwd_up_gemm", "bwd_pointwise", "bwd_bias", "bwd_gu_gemm",
           "bwd_gh_gemm", "bwd_attention", "bwd_gw_gemm", "bwd_gx_gemm", "splitk_reduce", "emb_keys", "emb_sort",
           "emb_reduce", "gather_q8", "quantize", "head_gate", "head_fwd_gemm", "head_out", "head_loss",
           "head_out_bwd", "head_gw_gemm", "head_gx_gemm", "head_gate_bwd", "head_colsum", "emb_fused"]
MAX_HIDDEN = 8


class RdcnConfig(ctypes.Structure):
    _fields_ = [("batch_max", ctypes.c_int64), ("num_cat", ctypes.c_int32), ("emb_dim", ctypes.c_int32),
                ("num_dense", ctypes.c_int32), ("rank", ctypes.c_int32), ("num_layers", ctypes.c_int32),
                ("qr_rows_q", ctypes.c_int32), ("qr_rows_r", ctypes.c_int32), ("combine", ctypes.c_int32),
                ("multi_hot", ctypes.c_int32), ("id_type", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("activation_mode", ctypes.c_int32), ("vocab", ctypes.c_int64), ("attn_alpha", ctypes.c_float),
                ("skip_beta", ctypes.c_float), ("temperature", ctypes.c_float), ("parallel_branch", ctypes.c_int32),
                ("hashed", ctypes.c_int32), ("reserved2", ctypes.c_int32), ("hash_seed", ctypes.c_uint64)]


class RdcnWeights(ctypes.Structure):
    _fields_ = [("w_down", ctypes.c_void_p * MAX_LAYERS), ("u", ctypes.c_void_p * MAX_LAYERS),
                ("bias", ctypes.c_void_p * MAX_LAYERS)]


class RdcnHeadConfig(ctypes.Structure):
    _fields_ = [("num_hidden", ctypes.c_int32), ("hidden", ctypes.c_int32 * MAX_HIDDEN), ("gated", ctypes.c_int32),
                ("num_buckets", ctypes.c_int32), ("bucket_lo", ctypes.c_float), ("bucket_step", ctypes.c_float)]


class RdcnHeadWeights(ctypes.Structure):
    _fields_ = [("w", ctypes.c_void_p * MAX_HIDDEN), ("b", ctypes.c_void_p * MAX_HIDDEN),
                ("gate_w", ctypes.c_void_p * MAX_HIDDEN), ("gate_b", ctypes.c_void_p * MAX_HIDDEN),
                ("w_out", ctypes.c_void_p), ("b_out", ctypes.c_void_p), ("cal_w", ctypes.c_void_p),
                ("cal_b", ctypes.c_void_p)]


def make_head_config(hidden: Sequence[int], gated: bool, num_buckets: int, bucket_lo: float,
                     bucket_step: float) -> RdcnHeadConfig:
    c = RdcnHeadConfig()
    c.num_hidden = len(hidden)
    for i, n in enumerate(hidden):
        c.hidden[i] = n
    c.gated, c.num_buckets, c.bucket_lo, c.bucket_step = int(gated), num_buckets, bucket_lo, bucket_step
    return c


def head_weights(p: dict) -> RdcnHeadWeights:
    """p: W, b, (G, c), w_out, b_out, cal_w, cal_b (device tensors; G and c only when gated)."""
    w = RdcnHeadWeights()
    for l in range(len(p["W"])):
        w.w[l], w.b[l] = p["W"][l].data_ptr(), p["b"][l].data_ptr()
        if p.get("G") is not None:
            w.gate_w[l], w.gate_b[l] = p["G"][l].data_ptr(), p["c"][l].data_ptr()
    w.w_out, w.b_out = p["w_out"].data_ptr(), p["b_out"].data_ptr()
    w.cal_w, w.cal_b = p["cal_w"].data_ptr(), p["cal_b"].data_ptr()
    return w


class RdcnError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__("%s failed: %s (%d)" % (fn, status_string(status), status))


_lib = None


def load(build_if_missing: bool = True):
    """Load librdcn.so (building it first if absent)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        if not build_if_missing:
            raise RuntimeError("librdcn.so is not built (%s)" % LIB_PATH)
        from . import build_lib
        build_lib.build()
    L = ctypes.CDLL(LIB_PATH)
    vp, i64, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t
    st = ctypes.c_int
    L.rdcn_status_string.argtypes = [st]
    L.rdcn_status_string.restype = ctypes.c_char_p
    L.rdcn_create.argtypes = [ctypes.POINTER(RdcnConfig), ctypes.POINTER(vp)]
    L.rdcn_destroy.argtypes = [vp]
    L.rdcn_dim.argtypes = [vp, ctypes.POINTER(i64)]
    L.rdcn_workspace_bytes.argtypes = [vp, i64, ctypes.POINTER(sz), ctypes.POINTER(sz)]
    L.qr_embed_gather.argtypes = [vp, i64, vp, vp, vp, vp, vp, vp, vp]
    L.qr_quantize_tables.argtypes = [vp, i64, vp, vp, vp, vp]
    L.qr_embed_gather_q8.argtypes = [vp, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    L.qr_embed_backward_workspace.argtypes = [vp, i64, i64, ctypes.POINTER(sz)]
    L.qr_embed_backward.argtypes = [vp, i64, i64, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.qr_embed_backward_static.argtypes = [vp, i64, i64, vp, vp, vp, vp, vp, vp, vp, vp]
    L.rdcn_forward.argtypes = [vp, i64, vp, ctypes.POINTER(RdcnWeights), vp, vp, vp, vp]
    L.rdcn_backward.argtypes = [vp, i64, vp, ctypes.POINTER(RdcnWeights), vp, vp, vp, ctypes.POINTER(RdcnWeights),
                                vp, vp]
    L.rdcn_check_device_errors.argtypes = [vp, vp]
    L.rdcn_head_configure.argtypes = [vp, ctypes.POINTER(RdcnHeadConfig)]
    L.rdcn_head_workspace_bytes.argtypes = [vp, i64, ctypes.POINTER(sz), ctypes.POINTER(sz)]
    L.rdcn_head_forward.argtypes = [vp, i64, vp, vp, ctypes.POINTER(RdcnHeadWeights), vp, vp, vp, vp]
    L.rdcn_head_logloss.argtypes = [vp, i64, vp, vp, ctypes.c_float, vp, vp, vp]
    L.rdcn_head_backward.argtypes = [vp, i64, vp, vp, ctypes.POINTER(RdcnHeadWeights), vp, vp, vp, vp,
                                     ctypes.POINTER(RdcnHeadWeights), vp, vp]
    L.rdcn_profile_start.argtypes = [vp, ctypes.c_int32, ctypes.c_uint32]
    L.rdcn_set_side_stream.argtypes = [vp, ctypes.c_int32]
    L.rdcn_profile_stop.argtypes = [vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]
    for name in EXPORTS:
        if name != "rdcn_status_string":
            getattr(L, name).restype = st
    _lib = L
    return L


def status_string(s: int) -> str:
    return load().rdcn_status_string(s).decode()


def _check(fn: str, s: int):
    if s != RDCN_OK:
        raise RdcnError(fn, s)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def make_config(batch_max: int, num_cat: int, emb_dim: int, num_dense: int, rank: int, num_layers: int,
                qr_rows_q: int, qr_rows_r: int, vocab: int, combine: str = "sum", multi_hot: bool = False,
                id_type: str = "i64", dtype: str = "bf16", attn_alpha: float = 0.0, skip_beta: float = 1.0,
                temperature: float = 1.0, activation_mode: str = "storage",
                parallel_branch: bool = False, hashed: bool = False, hash_seed: int = 0) -> RdcnConfig:
    c = RdcnConfig()
    c.batch_max, c.num_cat, c.emb_dim, c.num_dense = batch_max, num_cat, emb_dim, num_dense
    c.rank, c.num_layers, c.qr_rows_q, c.qr_rows_r = rank, num_layers, qr_rows_q, qr_rows_r
    c.combine = COMBINE_MUL if combine == "mul" else COMBINE_SUM
    c.multi_hot = int(multi_hot)
    c.id_type = I64 if id_type == "i64" else I32
    c.dtype = BF16 if dtype == "bf16" else F32
    c.vocab = vocab
    c.attn_alpha, c.skip_beta, c.temperature = attn_alpha, skip_beta, temperature
    c.activation_mode = ACT_MODES[activation_mode]
    c.parallel_branch = int(parallel_branch)
    c.hashed = int(hashed)
    c.hash_seed = hash_seed
    return c


def config_for(wl, batch_max: Optional[int] = None, id_type: str = "i64") -> RdcnConfig:
    """Config of a synthetic workload (paper_2402_06859_amd.synth.Workload)."""
    return make_config(batch_max or wl.batch, wl.num_cat, wl.emb_dim, wl.num_dense, wl.rank, wl.num_layers,
                       wl.table_rows, wl.table_rows, 0 if wl.hashed else wl.vocab, wl.combine, wl.multi_hot, id_type,
                       wl.dtype, wl.alpha, wl.beta, wl.temperature, wl.act_mode, wl.parallel, wl.hashed,
                       wl.hash_seed)


def _weights(w_down: Sequence[torch.Tensor], u: Sequence[torch.Tensor], bias: Sequence[torch.Tensor]) -> RdcnWeights:
    w = RdcnWeights()
    for l, (a, b, c) in enumerate(zip(w_down, u, bias)):
        w.w_down[l], w.u[l], w.bias[l] = a.data_ptr(), b.data_ptr(), c.data_ptr()
    return w


class Rdcn:
    """One librdcn handle. Tensors are CUDA (HIP) tensors, contiguous, in the documented layouts."""

    def __init__(self, cfg: RdcnConfig):
        L = load()
        self.cfg = cfg
        h = ctypes.c_void_p()
        _check("rdcn_create", L.rdcn_create(ctypes.byref(cfg), ctypes.byref(h)))
        self.h = h
        d = ctypes.c_int64()
        _check("rdcn_dim", L.rdcn_dim(h, ctypes.byref(d)))
        self.d = d.value

    def close(self):
        if getattr(self, "h", None) is not None and self.h.value:
            load().rdcn_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---- workspace
    def workspace_bytes(self, batch: int):
        s, t = ctypes.c_size_t(), ctypes.c_size_t()
        _check("rdcn_workspace_bytes", load().rdcn_workspace_bytes(self.h, batch, ctypes.byref(s), ctypes.byref(t)))
        return s.value, t.value

    def embed_backward_workspace(self, batch: int, nnz: int) -> int:
        s = ctypes.c_size_t()
        _check("qr_embed_backward_workspace", load().qr_embed_backward_workspace(self.h, batch, nnz, ctypes.byref(s)))
        return s.value

    # ---- entry points
    def qr_embed_gather(self, batch, ids, offsets, q_tables, r_tables, dense, x0, stream=None):
        _check("qr_embed_gather", load().qr_embed_gather(self.h, batch, _ptr(ids), _ptr(offsets), _ptr(q_tables),
                                                         _ptr(r_tables), _ptr(dense), _ptr(x0), _stream(stream)))

    def qr_quantize_tables(self, rows, tables, codes, params, stream=None):
        _check("qr_quantize_tables", load().qr_quantize_tables(self.h, rows, _ptr(tables), _ptr(codes), _ptr(params),
                                                               _stream(stream)))

    def qr_embed_gather_q8(self, batch, ids, offsets, q_codes, q_params, r_codes, r_params, dense, x0, stream=None):
        _check("qr_embed_gather_q8", load().qr_embed_gather_q8(
            self.h, batch, _ptr(ids), _ptr(offsets), _ptr(q_codes), _ptr(q_params), _ptr(r_codes), _ptr(r_params),
            _ptr(dense), _ptr(x0), _stream(stream)))

    def qr_embed_backward(self, batch, nnz, ids, offsets, q_tables, r_tables, grad_x0, grad_q, grad_r, scratch,
                          stream=None):
        _check("qr_embed_backward", load().qr_embed_backward(
            self.h, batch, nnz, _ptr(ids), _ptr(offsets), _ptr(q_tables), _ptr(r_tables), _ptr(grad_x0),
            _ptr(grad_q), _ptr(grad_r), _ptr(scratch), scratch.numel() * scratch.element_size(), _stream(stream)))

    def qr_embed_backward_static(self, batch, nnz, ids, offsets, q_tables, r_tables, grad_x0, grad_q, grad_r,
                                 stream=None):
        _check("qr_embed_backward_static", load().qr_embed_backward_static(
            self.h, batch, nnz, _ptr(ids), _ptr(offsets), _ptr(q_tables), _ptr(r_tables), _ptr(grad_x0),
            _ptr(grad_q), _ptr(grad_r), _stream(stream)))

    def rdcn_forward(self, batch, x0, w_down, u, bias, x_out, saved, scratch=None, stream=None):
        w = _weights(w_down, u, bias)
        _check("rdcn_forward", load().rdcn_forward(self.h, batch, _ptr(x0), ctypes.byref(w), _ptr(x_out), _ptr(saved),
                                                   _ptr(scratch), _stream(stream)))

    def rdcn_backward(self, batch, x0, w_down, u, bias, saved, grad_out, grad_x0, g_w_down, g_u, g_bias, scratch,
                      stream=None):
        w = _weights(w_down, u, bias)
        g = _weights(g_w_down, g_u, g_bias)
        _check("rdcn_backward", load().rdcn_backward(self.h, batch, _ptr(x0), ctypes.byref(w), _ptr(saved),
                                                     _ptr(grad_out), _ptr(grad_x0), ctypes.byref(g), _ptr(scratch),
                                                     _stream(stream)))

    # ---- head (layers after the cross stack)
    def head_configure(self, cfg: RdcnHeadConfig):
        _check("rdcn_head_configure", load().rdcn_head_configure(self.h, ctypes.byref(cfg)))
        self.head_cfg = cfg

    def head_workspace_bytes(self, batch: int):
        s, t = ctypes.c_size_t(), ctypes.c_size_t()
        _check("rdcn_head_workspace_bytes",
               load().rdcn_head_workspace_bytes(self.h, batch, ctypes.byref(s), ctypes.byref(t)))
        return s.value, t.value

    def head_forward(self, batch, x, e_cal, params: dict, y_logit, y_cal, saved, stream=None):
        w = head_weights(params)
        _check("rdcn_head_forward", load().rdcn_head_forward(self.h, batch, _ptr(x), _ptr(e_cal), ctypes.byref(w),
                                                             _ptr(y_logit), _ptr(y_cal), _ptr(saved),
                                                             _stream(stream)))

    def head_logloss(self, batch, y_cal, labels, scale, loss=None, grad=None, stream=None):
        _check("rdcn_head_logloss", load().rdcn_head_logloss(self.h, batch, _ptr(y_cal), _ptr(labels), scale,
                                                             _ptr(loss), _ptr(grad), _stream(stream)))

    def head_backward(self, batch, x, e_cal, params: dict, saved, grad_ycal, grad_x, grad_e, grads: dict, scratch,
                      stream=None):
        w = head_weights(params)
        g = head_weights(grads)
        _check("rdcn_head_backward", load().rdcn_head_backward(
            self.h, batch, _ptr(x), _ptr(e_cal), ctypes.byref(w), _ptr(saved), _ptr(grad_ycal), _ptr(grad_x),
            _ptr(grad_e), ctypes.byref(g), _ptr(scratch), _stream(stream)))

    def profile_start(self, max_launches: int = 8192, kernels=None):
        """Time the launches of `kernels` (names from KERNELS; all when None)."""
        mask = 0xFFFFFFFF if kernels is None else sum(1 << KERNELS.index(k) for k in kernels)
        _check("rdcn_profile_start", load().rdcn_profile_start(self.h, max_launches, mask))

    def profile_stop(self) -> dict:
        """{kernel: (total_ms, launches)} of the launches timed since profile_start."""
        n = len(KERNELS)
        ms = (ctypes.c_double * n)()
        cnt = (ctypes.c_int64 * n)()
        _check("rdcn_profile_stop", load().rdcn_profile_stop(self.h, ms, cnt))
        return {k: (ms[i], cnt[i]) for i, k in enumerate(KERNELS)}

    def set_side_stream(self, enable: bool):
        """Run the backward's weight-gradient work on the handle's second stream (default) or not."""
        _check("rdcn_set_side_stream", load().rdcn_set_side_stream(self.h, int(enable)))

    def check_device_errors(self, stream=None) -> int:
        """Synchronise and return (and clear) the device error status (RDCN_OK, RDCN_ERR_INDEX or
        RDCN_ERR_RANGE)."""
        return load().rdcn_check_device_errors(self.h, _stream(stream))
