"""The whole training step captured in a HIP graph (torch.cuda.CUDAGraph) replays
bit-identically to the eager step.

The library's calls issue kernel launches only (no memsets, copies or host
synchronisation), so a caller can capture a step once and replay it. Each replay
here is followed by eager work on the same buffers and compared with the eager
result, several times in a row (replays after the first must not differ).
"""
import pytest
import torch

from gpu_helpers import need_gpu
from paper_2402_06859_amd.step import DeviceBatch, DeviceHead
from paper_2402_06859_amd.synth import HEADS, WORKLOADS, make_head_inputs, make_inputs

pytestmark = pytest.mark.gpu


def _outputs(db, dh=None):
    outs = [db.x0, db.x_out, db.grad_x0, db.grad_q, db.grad_r] + db.g_w_down + db.g_u + db.g_bias
    if dh is not None:
        outs += [dh.y, dh.y_cal, dh.loss, dh.g_cal, dh.grad_x, dh.grad_e, dh.grads["w_out"], dh.grads["cal_w"]]
        outs += dh.grads["W"] + dh.grads["b"] + dh.grads["G"]
    return [t.clone() for t in outs]


def _same(a, b):
    for x, y in zip(a, b):
        xv = x.view(torch.int16) if x.dtype == torch.bfloat16 else x
        yv = y.view(torch.int16) if y.dtype == torch.bfloat16 else y
        if not torch.equal(xv, yv):
            return False
    return True


@pytest.mark.parametrize("with_head", [False, True])
def test_step_graph_replays_match_eager(with_head):
    need_gpu()
    wl = WORKLOADS["small"].with_(batch=1024)
    print("graph step", wl.name, "B", wl.batch, "head", with_head, flush=True)
    db = DeviceBatch(wl, make_inputs(wl, bias_std=0.1))
    dh = DeviceHead(db.lib, HEADS["small"], make_head_inputs(wl, HEADS["small"], with_x=False), wl.batch) \
        if with_head else None

    def step():
        db.grad_q.zero_()  # table gradients accumulate: start each step from zero
        db.grad_r.zero_()
        if dh is None:
            db.step()
        else:
            dh.tower_step(db)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()  # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    step()
    torch.cuda.synchronize()
    eager = _outputs(db, dh)

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for i in range(3):
        db.x_out.zero_()  # make stale results visible
        db.grad_x0.fill_(1.0)
        graph.replay()
        torch.cuda.synchronize()
        assert _same(_outputs(db, dh), eager), "replay %d differs from the eager step" % i
        step()  # eager work between replays
        torch.cuda.synchronize()
        assert _same(_outputs(db, dh), eager)
