"""Device buffers for one synthetic batch and the sequence of librdcn calls that
make one training step of the path: gather -> forward -> backward -> embedding
backward. Only allocation and call order live here; all arithmetic is in the
library's kernels.
"""
from __future__ import annotations

from typing import Optional

import torch

from .rdcn import Rdcn, config_for
from .synth import Workload

_DT = {"bf16": torch.bfloat16, "f32": torch.float32}


class DeviceBatch:
    def __init__(self, wl: Workload, inp: dict, device: str = "cuda", id_type: str = "i64",
                 batch_max: Optional[int] = None):
        self.wl = wl
        self.B = inp["batch"]
        dev = torch.device(device)
        dt = _DT[wl.dtype]
        self.lib = Rdcn(config_for(wl, batch_max or self.B, id_type))
        d = self.lib.d
        assert d == wl.d
        ids = inp["ids"]
        self.ids = (ids if id_type == "i64" else ids.to(torch.int32)).contiguous().to(dev)
        self.offsets = None if inp["offsets"] is None else inp["offsets"].contiguous().to(dev)
        self.nnz = int(ids.numel())
        self.q_tables = inp["q_tables"].contiguous().to(dev)
        self.r_tables = inp["r_tables"].contiguous().to(dev)
        self.dense = inp["dense"].contiguous().to(dev)
        self.w_down = [w.contiguous().to(dev) for w in inp["w_down"]]
        self.u = [w.contiguous().to(dev) for w in inp["u"]]
        self.bias = [w.contiguous().to(dev) for w in inp["bias"]]
        self.grad_out = inp["grad_out"].contiguous().to(dev) if "grad_out" in inp else None
        B = self.B
        self.x0 = torch.empty((B, d), dtype=dt, device=dev)
        self.x_out = torch.empty((B, d), dtype=dt, device=dev)
        saved_b, scratch_b = self.lib.workspace_bytes(B)
        self.saved = torch.empty(max(saved_b, 1), dtype=torch.uint8, device=dev)
        self.scratch = torch.empty(max(scratch_b, 1), dtype=torch.uint8, device=dev)
        self.grad_x0 = torch.empty((B, d), dtype=torch.float32, device=dev)
        self.g_w_down = [torch.empty(w.shape, dtype=torch.float32, device=dev) for w in self.w_down]
        self.g_u = [torch.empty(w.shape, dtype=torch.float32, device=dev) for w in self.u]
        self.g_bias = [torch.empty(w.shape, dtype=torch.float32, device=dev) for w in self.bias]
        self.grad_q = torch.zeros(self.q_tables.shape, dtype=torch.float32, device=dev)
        self.grad_r = torch.zeros(self.r_tables.shape, dtype=torch.float32, device=dev)
        eb = self.lib.embed_backward_workspace(B, self.nnz)
        self.emb_scratch = torch.empty(max(eb, 1), dtype=torch.uint8, device=dev)

    # individual calls
    def gather(self, stream=None):
        self.lib.qr_embed_gather(self.B, self.ids, self.offsets, self.q_tables, self.r_tables, self.dense, self.x0,
                                 stream)

    def forward(self, stream=None):
        self.lib.rdcn_forward(self.B, self.x0, self.w_down, self.u, self.bias, self.x_out, self.saved, self.scratch,
                              stream)

    def backward(self, grad_out: Optional[torch.Tensor] = None, stream=None):
        g = self.grad_out if grad_out is None else grad_out
        self.lib.rdcn_backward(self.B, self.x0, self.w_down, self.u, self.bias, self.saved, g, self.grad_x0,
                               self.g_w_down, self.g_u, self.g_bias, self.scratch, stream)

    def embed_backward(self, grad_x0: Optional[torch.Tensor] = None, stream=None):
        self.lib.qr_embed_backward(self.B, self.nnz, self.ids, self.offsets, self.q_tables, self.r_tables,
                                   self.grad_x0 if grad_x0 is None else grad_x0, self.grad_q, self.grad_r,
                                   self.emb_scratch, stream)

    def step(self, stream=None):
        """One pass of the whole path (table gradients accumulate)."""
        self.gather(stream)
        self.forward(stream)
        self.backward(stream=stream)
        self.embed_backward(stream=stream)


class DeviceHead:
    """Device buffers of the head after the cross stack (gated MLP, logit, isotonic
    calibration, log loss) on the handle `lib`, and its call order."""

    def __init__(self, lib: Rdcn, head, hinp: dict, B: int, device: str = "cuda"):
        from .rdcn import make_head_config
        dev = torch.device(device)
        self.lib = lib
        self.head = head
        self.B = B
        lib.head_configure(make_head_config(head.widths, head.gated, head.buckets, head.lo, head.step))
        keys = ["W", "b"] + (["G", "c"] if head.gated else [])
        self.params = {k: [t.contiguous().to(dev) for t in hinp[k]] for k in keys}
        for k in ("w_out", "b_out", "cal_w", "cal_b"):
            self.params[k] = hinp[k].contiguous().to(dev)
        self.e = hinp["e"].contiguous().to(dev)
        self.labels = hinp["labels"].contiguous().to(dev)
        self.g_cal_in = hinp["g_cal"].contiguous().to(dev) if "g_cal" in hinp else None
        self.x = hinp["x"].contiguous().to(dev) if "x" in hinp else None
        saved_b, scratch_b = lib.head_workspace_bytes(B)
        self.saved = torch.empty(max(saved_b, 1), dtype=torch.uint8, device=dev)
        self.scratch = torch.empty(max(scratch_b, 1), dtype=torch.uint8, device=dev)
        self.y = torch.empty(B, dtype=torch.float32, device=dev)
        self.y_cal = torch.empty(B, dtype=torch.float32, device=dev)
        self.loss = torch.empty(B, dtype=torch.float32, device=dev)
        self.g_cal = torch.empty(B, dtype=torch.float32, device=dev)
        self.grad_x = torch.empty((B, lib.d), dtype=torch.bfloat16, device=dev)
        self.grad_e = torch.empty(self.e.shape, dtype=torch.float32, device=dev)
        self.grads = {k: [torch.empty(t.shape, dtype=torch.float32, device=dev) for t in self.params[k]]
                      for k in keys}
        for k in ("w_out", "b_out", "cal_w", "cal_b"):
            self.grads[k] = torch.empty(self.params[k].shape, dtype=torch.float32, device=dev)

    def forward(self, x: Optional[torch.Tensor] = None, stream=None):
        self.lib.head_forward(self.B, self.x if x is None else x, self.e, self.params, self.y, self.y_cal,
                              self.saved, stream)

    def logloss(self, stream=None):
        """Mean log loss over the batch: per-sample losses and dLoss/dy_cal = (sigmoid - label) / B."""
        self.lib.head_logloss(self.B, self.y_cal, self.labels, 1.0 / max(self.B, 1), self.loss, self.g_cal, stream)

    def backward(self, x: Optional[torch.Tensor] = None, g_cal: Optional[torch.Tensor] = None, stream=None):
        self.lib.head_backward(self.B, self.x if x is None else x, self.e, self.params, self.saved,
                               self.g_cal if g_cal is None else g_cal, self.grad_x, self.grad_e, self.grads,
                               self.scratch, stream)

    def tower_step(self, db: "DeviceBatch", stream=None):
        """One training step of a Feed-style tower: gather -> cross stack -> head ->
        log loss -> head backward -> cross-stack backward -> embedding backward."""
        db.gather(stream)
        db.forward(stream)
        self.forward(db.x_out, stream)
        self.logloss(stream)
        self.backward(db.x_out, stream=stream)
        db.backward(self.grad_x, stream)
        db.embed_backward(stream=stream)
