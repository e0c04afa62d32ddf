"""Benchmark: samples/s of one training step of the QR-embedding + Residual-DCN path.

One step = qr_embed_gather -> rdcn_forward -> rdcn_backward -> qr_embed_backward
on one synthetic batch already resident in HBM. The default workload is the
largest one that fits one GPU ("large": batch 32768, 200 single-hot features
QR-hashed into 4473 x 48 tables, 1024 dense features, d = 10624, 6 Residual-DCN
layers of rank 1024 with the attention term, bf16 weights and storage with float
accumulation, activations x_l and h held in f16).

Prints ONE JSON line. Besides throughput (timed over the steps alone, no
per-kernel events) it carries:
  roofline      -- the kernel with the largest share of a step: algorithmic work
                   per launch / average launch time, measured with HIP events on
                   the launch stream over as many steps again, run after the timed
                   region with every kernel alone on the stream
  cpu_baseline  -- the CPU oracle (oracle/: plain C loops) timed on this host on a
                   bounded sub-batch of the same workload, one process per core
  kernels, phases -- per-kernel average times and each against its own bound
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "samples/s fwd+bwd of QR-embed + Residual DCN stack; % bf16 MFMA peak; gather GB/s"
PEAK_BF16_TFLOPS = 2516.6   # dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # fp32 vector with packed (dual) FMA
# The kernels are built without packed fp32 instructions, so the attainable fp32
# vector rate is 256 CUs x 64 lanes x 2 flops x 2.4 GHz = 78.6 TFLOP/s of FMAs.
PEAK_F32_UNPACKED_TFLOPS = 78.6
PEAK_HBM_GBS = 8000.0
# Issue cost of one v_exp_f32 in FMA slots (measured on MI355X: an exp + add chain
# runs at ~14.7 T/s against ~39 T FMA slots/s, i.e. about two slots per exp).
EXP_SLOTS = 2.0
# Exponential rate of the chip: one wave-wide v_exp_f32 issues every 8 clocks per SIMD
# (measured: 8.1 clk; half the rate of a plain VALU op), so 256 CUs x 4 SIMDs x 8 lanes
# per clock x 2.4 GHz = 19.66 T exp/s. The attention kernels' roofline is this rate.
EXP_PEAK_PER_S = 256 * 4 * 8 * 2.4e9
# Measured rate of independent exp + add pairs over all CUs (an exponential and one
# more VALU op per pair, as a softmax needs at least): a practical ceiling beside the peak.
EXP_ADD_MEASURED_PER_S = 14.7e12
# Measured rates of the attention inner loop's instruction mix run alone (per lane: 16
# exponentials, 8 packed conversions to f16, one 32x32x8 and two 16x16x32 f16 MFMAs,
# 8 waves per SIMD), and of exponentials alone: what the exponent loop can reach
# without loads, barriers or per-sample set-up.
EXP_LOOP_MIX_MEASURED_PER_S = 13.5e12
EXP_ONLY_MEASURED_PER_S = 17.4e12


def kernel_work(wl, B: int) -> dict:
    """Algorithmic work of one launch of each kernel: (flops, bytes, alu_ops).

    bytes are the bytes the algorithm must move (each operand read once, each
    result written once); flops count a multiply-add as 2; alu_ops is the vector
    ALU work of the per-sample attention kernels in FMA-equivalent flops per
    (query, key) pair: the exponent argument (one FMA = 2), the exponential
    (EXP_SLOTS FMA slots = 4) and, for bf16 models whose sums run on the matrix
    cores, half a packed f16 conversion (1); their backward evaluates every pair
    once (the forward saved each row's normaliser). Float-storage models
    accumulate on the vector ALU instead (forward + 3 flops per pair; backward
    evaluates every pair twice, + 11 flops).
    """
    d, r, n = wl.d, wl.rank, wl.n_proj
    nr = n * r
    eb = 2 if wl.dtype == "bf16" else 4
    pb = 4 if wl.attention else eb  # [v|q|k] storage
    F, D, Nd = wl.num_cat, wl.emb_dim, wl.num_dense
    hot = wl.bag_mean if wl.multi_hot else 1.0
    L = wl.num_layers
    hr = wl.h_width          # width of the up projection's input
    dl = 2 if wl.parallel else 1  # launches of the down and gh GEMMs per layer (plain branch apart)
    w = {}
    tp = wl.table_pairs  # QR table pairs per feature (2 with the hashed front-end)
    # gather: ids, both table rows of every pair per id, x0 write, dense read
    w["gather"] = (0.0, B * (F * hot * 8 + 2 * tp * F * hot * D * eb + F * D * eb + 2 * Nd * eb), 0.0)
    w["fwd_down_gemm"] = (2.0 * B * nr * d / dl, (dl * B * d * eb + nr * d * eb + B * nr * pb) / dl, 0.0)
    exp_f = 2.0 * EXP_SLOTS
    pair_fwd = (2.0 + exp_f + 1.0) if wl.dtype == "bf16" else (2.0 + exp_f + 3.0)
    pair_bwd = (2.0 + exp_f + 1.0) if wl.dtype == "bf16" else (2 * (2.0 + exp_f) + 11.0)
    # saved per row by the matrix-core forward: (o, Z) and the backward's row sums (W1, W2)
    stats = 4 * r * 4 if wl.dtype == "bf16" else 0
    # h, and its second plane when the activations are held as f16 or as bf16 hi + lo
    h_out = r * eb * (2 if wl.act_mode in ("f16", "hilo") else 1)
    w["fwd_attention"] = (0.0, B * (3 * r * 4 + h_out + stats), pair_fwd * B * r * r)
    # up projection + cross epilogue: h, U, bias, x0, x_l in; t, x_{l+1} out. With hi + lo
    # activations x_l is read and x_{l+1} written as two planes; with f16 activations x_{l+1}
    # is written as f16 and as a bf16 copy (the weight gradient's operand).
    xl_planes = 2 if wl.act_mode == "hilo" else 1
    xo_planes = 2 if wl.act_mode in ("f16", "hilo") else 1
    w["fwd_up_gemm"] = (2.0 * B * d * hr,
                        B * hr * eb + d * hr * eb + d * eb + B * d * eb * (2 + xl_planes + xo_planes), 0.0)
    # average over layers of: g in (storage on the top layer, float below), x0, t, grad_x0 (rmw below top), gt out
    gin = (eb + (L - 1) * 4) / L
    gx = (4 + (L - 1) * 8) / L
    w["bwd_pointwise"] = (0.0, B * d * (gin + 2 * eb + gx + eb), 0.0)
    w["bwd_bias"] = (0.0, -(-B // 128) * d * 4 + d * 4, 0.0)
    w["bwd_gu_gemm"] = (2.0 * d * hr * B, B * d * eb + B * hr * eb + d * hr * 4, 0.0)
    w["bwd_gh_gemm"] = (2.0 * B * hr * d / dl, (dl * B * d * eb + d * hr * eb + B * hr * (4 if wl.attention else eb)) / dl,
                        0.0)
    w["bwd_attention"] = (0.0, B * (3 * r * 4 + r * 4 + stats + 3 * r * eb), pair_bwd * B * r * r)
    w["bwd_gw_gemm"] = (2.0 * nr * d * B, B * nr * eb + B * d * eb + nr * d * 4, 0.0)
    w["bwd_gx_gemm"] = (2.0 * B * d * nr, B * nr * eb + nr * d * eb + 2 * B * d * 4, 0.0)
    # embedding backward: nnz ids, 2 (key, occurrence) pairs of 4 + 4 bytes per id
    nnz = B * F * hot
    passes = _radix_passes(F * tp * (2 * wl.table_rows))
    w["emb_keys"] = (0.0, nnz * 8 + 2 * tp * nnz * 8 + (nnz * 4 if wl.multi_hot else 0), 0.0)
    w["emb_sort"] = (0.0, passes * 2 * tp * nnz * (4 + 8 + 8), 0.0)  # histogram read + scatter read/write per pass
    w["emb_reduce"] = (0.0, 2 * tp * nnz * (8 + D * 4) + 2 * tp * F * wl.table_rows * D * 8, 0.0)
    # one-kernel path: ids (and bag offsets), each feature's gradient slab once, every table row
    # read and written once (+ the other table once with the product combine); the per-occurrence
    # re-reads of gradient slices are served by L2
    w["emb_fused"] = (0.0, nnz * 8 + (B * F * 8 if wl.multi_hot else 0) + B * F * D * 4
                      + 2 * F * wl.table_rows * D * 8 + (2 * F * wl.table_rows * D * eb if wl.combine == "mul" else 0),
                      0.0)
    # serving gather from 8-bit tables: codes (1 byte per value) and each row's (middle, scale)
    w["gather_q8"] = (0.0, B * (F * hot * 8 + 2 * tp * F * hot * (D + 8) + F * D * eb + 2 * Nd * eb), 0.0)
    return w


def head_work(wl, head, B: int) -> dict:
    """Algorithmic work per launch of the head kernels (averaged over the launches of a
    step where layers differ): flops of the logical widths (the zero padding to a
    multiple of 8 is not counted), bytes of each operand read once and each result
    written once (bf16 activations, weights and G; float gate logits, logits and
    calibration data)."""
    n = [wl.d] + list(head.hidden)
    L = len(head.hidden)
    K = head.buckets
    lay = range(1, L + 1)
    w = {}
    w["head_gate"] = (0.0, sum(B * n[l - 1] * 2 + B * 4 for l in lay) / L, 0.0)
    w["head_fwd_gemm"] = (sum(2.0 * B * n[l] * n[l - 1] for l in lay) / L,
                          sum(B * n[l - 1] * 2 + n[l] * n[l - 1] * 2 + B * n[l] * 2 + n[l] * 2 for l in lay) / L, 0.0)
    w["head_out"] = (0.0, B * n[L] * 2 + B * K * 4 + 3 * B * 4, 0.0)
    w["head_loss"] = (0.0, 4 * B * 4, 0.0)
    w["head_out_bwd"] = (0.0, 2 * B * n[L] * 2 + 2 * B * K * 4 + 5 * B * 4, 0.0)
    w["head_gw_gemm"] = (sum(2.0 * n[l] * n[l - 1] * B for l in lay) / L,
                         sum(B * n[l] * 2 + B * n[l - 1] * 2 + n[l] * n[l - 1] * 4 for l in lay) / L, 0.0)
    # G_l W_l: G and W in, the layer below's activations in (l > 1), its G (or grad_x) out
    w["head_gx_gemm"] = (sum(2.0 * B * n[l - 1] * n[l] for l in lay) / L,
                         sum(B * n[l] * 2 + n[l] * n[l - 1] * 2 + (B * n[l - 1] * 2 if l > 1 else 0)
                             + B * n[l - 1] * 2 for l in lay) / L, 0.0)
    w["head_gate_bwd"] = (0.0, B * 4 * 3, 0.0)
    col = (B * n[L] * 2 + B * 4) + B * 4 + B * K * 4 + B * 4 + sum(B * n[l] * 2 + B * n[l - 1] * 2 + 2 * B * 4
                                                                  for l in lay)
    w["head_colsum"] = (0.0, col / (4 + 3 * L), 0.0)
    return w


def _radix_passes(maxkey: int) -> int:
    bits = max(1, int(maxkey).bit_length())
    return -(-bits // 10)


def roofline_for(name: str, work: tuple, avg_s: float, bf16: bool) -> dict:
    flops, nbytes, alu = work
    if bf16 and name in ("fwd_attention", "bwd_attention"):
        # exponential-bound: one exp per (query, key) pair; alu holds 7 FMA-equivalent flops per pair
        exps = alu / 7.0
        return {"bound": "exp", "achieved": exps / avg_s / 1e12, "peak": EXP_PEAK_PER_S / 1e12, "unit": "Texp/s"}
    if alu > 0:
        return {"bound": "alu", "achieved": alu / avg_s / 1e12, "peak": PEAK_F32_UNPACKED_TFLOPS, "unit": "TFLOP/s"}
    peak_f = PEAK_BF16_TFLOPS if bf16 else PEAK_F32_TFLOPS
    t_f = flops / (peak_f * 1e12)
    t_b = nbytes / (PEAK_HBM_GBS * 1e9)
    if flops > 0 and t_f >= t_b:
        return {"bound": "mfma", "achieved": flops / avg_s / 1e12, "peak": peak_f, "unit": "TFLOP/s"}
    return {"bound": "hbm", "achieved": nbytes / avg_s / 1e9, "peak": PEAK_HBM_GBS, "unit": "GB/s"}


# Source files whose text determines each kernel class (a counter reading is only
# valid for the code it was taken on).
KERNEL_SOURCES = {
    "fwd_attention": ["attention.hip", "device_common.h"],
    "bwd_attention": ["attention.hip", "device_common.h"],
    "gather": ["gather.hip", "device_common.h"],
    "bwd_pointwise": ["pointwise.hip", "device_common.h"],
    "emb_keys": ["embed_bwd.hip", "device_common.h"],
    "emb_sort": ["embed_bwd.hip", "device_common.h"],
    "emb_reduce": ["embed_bwd.hip", "device_common.h"],
    "emb_fused": ["embed_bwd.hip", "device_common.h"],
}
for _k in ("fwd_down_gemm", "fwd_up_gemm", "bwd_gu_gemm", "bwd_gh_gemm", "bwd_gw_gemm", "bwd_gx_gemm"):
    KERNEL_SOURCES[_k] = ["gemm.hip", "gemm.h", "device_common.h"]
for _k in ("head_fwd_gemm", "head_gw_gemm", "head_gx_gemm"):
    KERNEL_SOURCES[_k] = ["gemm.hip", "gemm.h", "device_common.h", "mlp_common.h"]
for _k in ("head_gate", "head_out", "head_loss", "head_out_bwd", "head_gate_bwd", "head_colsum"):
    KERNEL_SOURCES[_k] = ["head.hip", "head.h", "device_common.h", "mlp_common.h"]


def sources_sha256(kernel: str) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES.get(kernel, []):
        with open(os.path.join(ROOT, "paper_2402_06859_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` on `workload` from the counter summaries
    under profiles/ (lines 'traffic: {json}'), or None when there is none or the
    kernel's sources changed since the counters were taken."""
    import glob
    if kernel not in KERNEL_SOURCES:
        return None
    sha = sources_sha256(kernel)
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        with open(path) as fh:
            for line in fh:
                if not line.startswith("traffic: "):
                    continue
                rec = json.loads(line[len("traffic: "):])
                if rec.get("kernel") == kernel and rec.get("workload") == workload and rec.get("sha256") == sha:
                    return float(rec["bytes_per_launch"])
    return None


def profile_tag(wl, head=None) -> str:
    """The workload key of the counter records under profiles/: the workload's name, then
    the variant and the head (e.g. 'small+hashed', 'feed+lmlp')."""
    return (wl.name + ("+hashed" if wl.hashed else "") + ("+parallel" if wl.parallel else "")
            + ("+" + head.name if head is not None else ""))


def counter_record(prefix: str, kernel: str, workload: str):
    """The '<prefix>: {json}' record of `kernel` on `workload` under profiles/ taken on the
    kernel's current sources, or None."""
    import glob
    if kernel not in KERNEL_SOURCES:
        return None
    sha = sources_sha256(kernel)
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        with open(path) as fh:
            for line in fh:
                if line.startswith(prefix + ": "):
                    rec = json.loads(line[len(prefix) + 2:])
                    if rec.get("kernel") == kernel and rec.get("workload") == workload and rec.get("sha256") == sha:
                        return rec
    return None


def phase_rooflines(work: dict, prof: dict, bf16: bool) -> dict:
    """Every timed kernel against its own bound: {kernel: {bound, achieved, unit, frac}}."""
    out = {}
    for k, (ms, n) in prof.items():
        if not n or k not in work:
            continue
        r = roofline_for(k, work[k], ms / n / 1e3, bf16)
        out[k] = {"bound": r["bound"], "achieved": r["achieved"], "unit": r["unit"], "frac": r["achieved"] / r["peak"]}
    return out


def gather_counter_gbps(tag: str, prof: dict):
    """HBM bytes of the gather from the FETCH_SIZE / WRITE_SIZE summaries under profiles/
    (while its sources are unchanged) over its measured launch time; None without a
    matching counter record."""
    t = measured_traffic("gather", tag)
    ms, n = prof.get("gather", (0.0, 0))
    return t / (ms / n / 1e3) / 1e9 if (t is not None and n) else None


def mfma_counter_rates(wl, tag: str, prof: dict) -> dict:
    """Matrix-core flops per launch of each GEMM phase from the MFMA counter summaries
    under profiles/ (lines 'mfma: {json}' with SQ_INSTS_VALU_MFMA_MOPS_BF16 / _F16 x 512
    flops, while the GEMM sources are unchanged) over the phase's measured launch time:
    {phase: {"tflops", "frac", "busy"}} (busy: SQ_VALU_MFMA_BUSY_CYCLES over SQ_BUSY_CU_CYCLES
    when recorded)."""
    import glob
    out = {}
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        with open(path) as fh:
            for line in fh:
                if not line.startswith("mfma: "):
                    continue
                rec = json.loads(line[len("mfma: "):])
                k = rec.get("kernel")
                if rec.get("workload") != tag or k not in KERNEL_SOURCES or rec.get("sha256") != sources_sha256(k):
                    continue
                ms, n = prof.get(k, (0.0, 0))
                if not n:
                    continue
                tf = rec["flops_per_launch"] / (ms / n / 1e3) / 1e12
                out[k] = {"tflops": tf, "frac": tf / PEAK_BF16_TFLOPS, "busy": rec.get("mfma_busy")}
    return out


def attention_exp_rate(wl, tag: str, B: int, prof: dict):
    """Exponentials per second of the attention kernels (one per (query, key) pair in the
    forward and one in the backward) against the chip's exponential rate and against the
    measured exp + add rate."""
    if not wl.attention:
        return None
    out = {}
    for k in ("fwd_attention", "bwd_attention"):
        ms, n = prof.get(k, (0.0, 0))
        if n:
            rate = B * wl.rank * wl.rank / (ms / n / 1e3)
            out[k] = {"exp_per_s": rate, "frac_of_peak": rate / EXP_PEAK_PER_S,
                      "frac_of_measured_exp_add_rate": rate / EXP_ADD_MEASURED_PER_S,
                      "frac_of_measured_loop_mix_rate": rate / EXP_LOOP_MIX_MEASURED_PER_S}
            rec = counter_record("trans", k, tag)
            if rec is not None:  # SQ_INSTS_VALU_TRANS_F32 x 64 of the same kernel and workload
                out[k]["counter_exps_per_launch"] = rec["exps_per_launch"]
                out[k]["counter_exps_over_pairs"] = rec["exps_per_launch"] / (B * wl.rank * wl.rank)
                out[k]["valu_instr_per_exp_lane"] = rec["valu_instr_per_launch"] * 64 / rec["exps_per_launch"]
    return out


def host_info() -> dict:
    """The host's logical CPU count, CPU model and available memory (for the CPU baseline)."""
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    avail = None
    try:
        with open("/proc/meminfo") as fh:
            for line in fh:
                if line.startswith("MemAvailable:"):
                    avail = int(line.split()[1]) * 1024
                    break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "cpu_model": model, "mem_available_bytes": avail}


def oracle_worker_bytes(wl) -> float:
    """Host memory one oracle process needs: the weights and their gradients in float64 (the
    C oracle's working copies), the storage-type and float32 copies of the inputs, and the
    tables (an upper estimate; the large workload measured 6.4 GB for 8.4 GB estimated)."""
    d, r, n, L = wl.d, wl.rank, wl.n_proj, wl.num_layers
    params = L * (n * r * d + d * wl.h_width + d)
    tables = 2 * wl.table_pairs * wl.num_cat * wl.table_rows * wl.emb_dim
    return params * (8 * 2 + 4 + 2 + 8) + tables * 14 + (1 << 30)


def _oracle_proc(wl, rows: int, head, seed: int, barrier, queue) -> None:
    """One baseline worker: draw its inputs, wait for the others, then time its oracle step
    (start and end on the system-wide monotonic clock)."""
    from threadpoolctl import threadpool_limits
    with threadpool_limits(limits=1):
        state = _oracle_prepare(wl, rows, head, seed)
        barrier.wait()
        t0 = time.perf_counter()
        _oracle_run(state)
        queue.put((t0, time.perf_counter()))


def cpu_baseline(wl, target_s: float, head=None) -> dict:
    """The oracle (oracle/: plain C loops, single-threaded, plus numpy float64 for a head)
    timed on this host: one step = gather + forward + backward (which recomputes its
    forward) + embedding backward on a sub-batch, in one single-threaded process per
    host core (at most 16, and no more than half the available memory holds). Each
    worker's sub-batch is sized from a single-threaded probe (8 rows, or 1 row on
    workloads with more than 2e7 cross-stack weights) to about `target_s` seconds. The
    workers draw their inputs, wait for each other, then time their steps; the value is
    the total rows over the span from the first start to the last end, and
    `single_thread_value` is the workers' mean own rate."""
    import multiprocessing as mp
    from threadpoolctl import threadpool_limits
    info = host_info()
    per_worker = oracle_worker_bytes(wl)
    workers = max(1, min(16, info["nproc"] or 1))
    if info["mem_available_bytes"]:
        workers = max(1, min(workers, int(0.5 * info["mem_available_bytes"] // per_worker)))
    probe = 1 if wl.d * wl.rank * wl.num_layers > 2e7 else 8
    with threadpool_limits(limits=1):
        t = _oracle_step(wl, probe, head)
    rows = int(max(1, min(wl.batch, round(probe * target_s / max(t, 1e-6)))))
    ctx = mp.get_context("spawn")
    barrier, queue = ctx.Barrier(workers), ctx.Queue()
    procs = [ctx.Process(target=_oracle_proc, args=(wl, rows, head, i, barrier, queue)) for i in range(workers)]
    for p in procs:
        p.start()
    spans = [queue.get() for _ in procs]
    for p in procs:
        p.join()
        if p.exitcode != 0:
            raise RuntimeError("oracle baseline worker failed (exit code %s)" % p.exitcode)
    wall = max(e for _, e in spans) - min(b for b, _ in spans)
    times = [e - b for b, e in spans]
    return {"value": workers * rows / wall, "unit": "samples/s", "cores": workers, "kind": "oracle",
            "sample": "%d processes x %d sample%s of the %s workload (gather + forward + backward + embedding "
                      "backward%s), %.1f s wall, one single-threaded oracle per core"
                      % (workers, rows, "" if rows == 1 else "s", wl.name, " + head" if head is not None else "",
                         wall),
            "single_thread_value": rows / (sum(times) / len(times)),
            "nproc": info["nproc"], "cpu_model": info["cpu_model"],
            "worker_memory_bytes_estimate": per_worker}


def _oracle_step(wl, rows: int, head=None, seed=None) -> float:
    return _oracle_run(_oracle_prepare(wl, rows, head, seed))


def _oracle_prepare(wl, rows: int, head=None, seed=None) -> dict:
    """Inputs of one oracle step (drawn, not timed)."""
    import oracle
    from paper_2402_06859_amd.synth import make_inputs
    oracle.lib()  # load the C oracle before anything is timed
    inp = make_inputs(wl, batch=rows, bias_std=0.0, seed=None if seed is None else 1000 + seed)
    W = [x.float().numpy() for x in inp["w_down"]]
    U = [x.float().numpy() for x in inp["u"]]
    b = [x.float().numpy() for x in inp["bias"]]
    if head is not None:
        from paper_2402_06859_amd.synth import make_head_inputs
        hinp = make_head_inputs(wl, head, batch=rows, with_x=False)
        f64 = lambda t: t.float().numpy().astype("float64")
        hp = {"W": [f64(w) for w in hinp["W"]], "b": [f64(v) for v in hinp["b"]], "w_out": f64(hinp["w_out"]),
              "b_out": float(hinp["b_out"].float()[0]), "cal_w": f64(hinp["cal_w"]), "cal_b": 0.0,
              "lo": head.lo, "step": head.step, "e": f64(hinp["e"])}
        if head.gated:
            hp["G"] = [f64(g) for g in hinp["G"]]
            hp["c"] = [float(c.float()[0]) for c in hinp["c"]]
        labels = f64(hinp["labels"])
    else:
        hp = labels = None
    return {"wl": wl, "rows": rows, "head": head, "inp": inp, "W": W, "U": U, "b": b, "hp": hp, "labels": labels}


def _oracle_run(state: dict) -> float:
    """Seconds of one oracle step: gather, forward, (head forward, loss and backward),
    backward (which recomputes its forward), embedding backward."""
    import oracle
    wl, rows, head, inp = state["wl"], state["rows"], state["head"], state["inp"]
    W, U, b, hp, labels = state["W"], state["U"], state["b"], state["hp"], state["labels"]
    F, D, Nd, m, bf16 = wl.num_cat, wl.emb_dim, wl.num_dense, wl.table_rows, wl.dtype == "bf16"
    t0 = time.perf_counter()
    if wl.hashed:
        x0 = oracle.gather_hashed(rows, F, D, Nd, m, m, wl.combine, bf16, wl.hash_seed, inp["ids"], inp["offsets"],
                                  inp["q_tables"], inp["r_tables"], inp["dense"])
    else:
        x0, _ = oracle.gather(rows, F, D, Nd, wl.vocab, m, m, wl.combine, bf16, inp["ids"], inp["offsets"],
                              inp["q_tables"], inp["r_tables"], inp["dense"])
    xL = oracle.forward(x0, W, U, b, wl.alpha, wl.beta, wl.temperature, parallel=wl.parallel)
    g_out = inp["grad_out"]
    if head is not None:
        from oracle import head as OH
        p = hp
        f = OH.head_forward(xL, p)
        _, g_cal = OH.logloss(f["y_cal"], labels)
        g_out = OH.head_backward(xL, p, g_cal / rows)["x"]
    gx0 = oracle.backward(x0, W, U, b, g_out, wl.alpha, wl.beta, wl.temperature, parallel=wl.parallel)[0]
    if wl.hashed:
        oracle.embed_backward_hashed(rows, F, D, Nd, m, m, wl.combine, wl.hash_seed, inp["ids"], inp["offsets"],
                                     inp["q_tables"], inp["r_tables"], gx0)
    else:
        oracle.embed_backward(rows, F, D, Nd, wl.vocab, m, m, wl.combine, inp["ids"], inp["offsets"],
                              inp["q_tables"], inp["r_tables"], gx0)
    return time.perf_counter() - t0


def time_graph_replays(step, steps: int, B: int) -> dict:
    """The step captured once in a HIP graph (torch.cuda.CUDAGraph; the library issues
    kernel launches only), then `steps` replays timed with events on the replay stream."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for _ in range(3):
        graph.replay()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        graph.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    return {"ms_per_step": ms, "samples_per_s": B / (ms / 1e3), "replays": steps}


def time_gather_q8(db, q8_bytes: float, bytes16: float, launches: int = 20) -> dict:
    """Serving-path gather from middle-max 8-bit tables (quantized once here), timed
    with HIP events on its launch stream; the storage-type gather on the same batch
    beside it."""
    import torch
    lib, D = db.lib, db.wl.emb_dim
    qs = []
    for t in (db.q_tables, db.r_tables):
        rows = t.numel() // D
        codes = torch.empty((rows, D), dtype=torch.int8, device=t.device)
        params = torch.empty((rows, 2), dtype=torch.float32, device=t.device)
        lib.qr_quantize_tables(rows, t, codes, params)
        qs += [codes, params]
    x0 = torch.empty_like(db.x0)
    res = {}
    for name in ("gather_q8", "gather"):
        lib.profile_start(launches, [name])
        for _ in range(launches):
            if name == "gather_q8":
                lib.qr_embed_gather_q8(db.B, db.ids, db.offsets, qs[0], qs[1], qs[2], qs[3], db.dense, x0)
            else:
                lib.qr_embed_gather(db.B, db.ids, db.offsets, db.q_tables, db.r_tables, db.dense, x0)
        ms, n = lib.profile_stop()[name]
        res[name] = ms / n * 1e3
    return {"avg_us": res["gather_q8"], "gbps": q8_bytes / (res["gather_q8"] * 1e-6) / 1e9,
            "table_bytes_per_value": 1, "storage_gather_avg_us": res["gather"],
            "storage_gather_gbps": bytes16 / (res["gather"] * 1e-6) / 1e9}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="large",
                    help="tiny, small, feed, multihot or large (the default: the largest single-GPU one)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="oracle time budget for cpu_baseline (0 = skip)")
    ap.add_argument("--side-stream", default="on", choices=["on", "off"],
                    help="run the backward's weight-gradient work on a second stream during the timed steps")
    ap.add_argument("--no-q8", action="store_true", help="skip the 8-bit serving-gather comparison")
    ap.add_argument("--id-mode", default="scatter", choices=["scatter", "rank"])
    ap.add_argument("--hashed", action="store_true",
                    help="Murmur-hashed front-end: raw ids hashed, two QR table pairs of 2^16 + 2^16 rows per feature")
    ap.add_argument("--parallel-branch", action="store_true",
                    help="plain and attention low-rank cross nets with their own weights in every layer")
    ap.add_argument("--head", default=None, metavar="NAME",
                    help="train a Feed-style tower: the cross stack's output goes through a head (lmlp: gated "
                         "4 x 3500 ReLU layers, logit, isotonic calibration, log loss) whose input gradient "
                         "drives the cross-stack backward")
    ap.add_argument("--graph", action="store_true",
                    help="also capture the step in a HIP graph and time its replays (graph_ms_per_step)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only copy MIB MiB device-to-device a few times (known traffic, to scale HBM counters)")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": n * 4, "copy_calibration_bytes_written": n * 4,
                          "launches": 3}), flush=True)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path; --gpus must be 1.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2402_06859_amd import rdcn
    from paper_2402_06859_amd.step import DeviceBatch, DeviceHead
    from paper_2402_06859_amd.synth import HEADS, WORKLOADS, make_head_inputs, make_inputs

    wl = WORKLOADS[args.workload]
    if args.parallel_branch:
        if not wl.attention:
            print("--parallel-branch needs a workload with the attention term", file=sys.stderr)
            sys.exit(2)
        wl = wl.with_(parallel=True)
    if args.hashed:
        wl = wl.with_(hashed=True, table_rows=1 << 16)
    head = HEADS[args.head] if args.head else None
    # the CPU baseline runs before anything touches the GPU (its worker processes are
    # started from a process that has not initialised it)
    cpu = cpu_baseline(wl, args.cpu_seconds, head) if args.cpu_seconds > 0 else None
    torch.cuda.set_device(0)
    inp = make_inputs(wl, id_mode=args.id_mode)
    db = DeviceBatch(wl, inp)
    B = db.B
    side_on = args.side_stream == "on"
    db.lib.set_side_stream(side_on)
    if head is not None:
        dh = DeviceHead(db.lib, head, make_head_inputs(wl, head, with_x=False), B)
        step = lambda: dh.tower_step(db)
    else:
        step = db.step
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if db.lib.check_device_errors() != rdcn.RDCN_OK:
        raise RuntimeError("device error flag raised during warm-up")

    # timed region: the steps alone, no per-kernel events
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = e0.elapsed_time(e1)
    if db.lib.check_device_errors() != rdcn.RDCN_OK:
        raise RuntimeError("device error flag raised during the timed steps")

    # per-kernel times, measured after the timed region with every kernel running alone
    # (the backward's weight-gradient work on the caller's stream): one step with events
    # around every launch finds the kernel with the largest share, then `steps` steps with
    # events around that kernel's launches only give its roofline
    db.lib.set_side_stream(False)
    db.lib.profile_start(4096)
    step()
    prof = db.lib.profile_stop()
    work = kernel_work(wl, B)
    if head is not None:
        work.update(head_work(wl, head, B))
    dominant = max((k for k in prof if k in work), key=lambda k: prof[k][0])
    # the gather (one launch per step) is timed over the same steps, not from one launch
    timed = [dominant] + (["gather"] if dominant != "gather" and prof.get("gather", (0, 0))[1] else [])
    db.lib.profile_start(4 * args.steps * 64, timed)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    steps_prof = db.lib.profile_stop()
    dom = steps_prof[dominant]
    db.lib.set_side_stream(side_on)

    ms_step = ms / args.steps
    avg_s = dom[0] / dom[1] / 1e3
    roof = roofline_for(dominant, work[dominant], avg_s, wl.dtype == "bf16")
    roof["frac"] = roof["achieved"] / roof["peak"]
    tag = profile_tag(wl, head)
    roof["traffic"] = measured_traffic(dominant, tag)
    roof["kernel"] = dominant
    roof["avg_us"] = avg_s * 1e6
    roof["launches"] = dom[1]
    roof["measured"] = "HIP events on the launch stream, %d steps after the timed region, kernels run alone" \
                       % args.steps
    if roof["bound"] == "exp":
        roof["frac_of_measured_exp_add_rate"] = roof["achieved"] * 1e12 / EXP_ADD_MEASURED_PER_S
        roof["frac_of_measured_loop_mix_rate"] = roof["achieved"] * 1e12 / EXP_LOOP_MIX_MEASURED_PER_S

    kernels = {k: {"avg_us": (v[0] / v[1] * 1e3) if v[1] else 0.0, "per_step": v[1]} for k, v in prof.items() if v[1]}
    gemm_flops = sum(work[k][0] * prof[k][1] for k in work if k.endswith("_gemm") and k in prof)
    gemm_s = sum(prof[k][0] for k in prof if k.endswith("_gemm")) / 1e3
    gprof = steps_prof.get("gather", (0.0, 0))
    if gprof[1]:
        prof["gather"] = gprof
        kernels["gather"] = {"avg_us": gprof[0] / gprof[1] * 1e3, "per_step": 1, "launches_timed": gprof[1]}
    gather_s = prof["gather"][0] / prof["gather"][1] / 1e3 if prof["gather"][1] else 0.0
    counter_gbps = gather_counter_gbps(profile_tag(wl, head), prof)
    out = {
        "metric": METRIC,
        "value": B * args.steps / (ms / 1e3),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "wall_ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded Zipf ids, N(0,1) dense, Xavier weights); inputs resident in HBM",
        "config": {"workload": workload_description(wl, B, head), "global_batch": B, "id_mode": args.id_mode,
                   "side_stream": args.side_stream},
        "roofline": roof,
        "gemm_mfma_frac": (gemm_flops / gemm_s / 1e12 / PEAK_BF16_TFLOPS) if gemm_s > 0 else None,
        "gemm_phases_tflops": {k: work[k][0] / (prof[k][0] / prof[k][1] / 1e3) / 1e12
                               for k in work if k.endswith("_gemm") and prof.get(k, (0, 0))[1]},
        "gather_hbm_frac": counter_gbps / PEAK_HBM_GBS if counter_gbps is not None else None,
        "gather_counter_gbps": counter_gbps,
        "gather_model_gbps": (work["gather"][1] / gather_s / 1e9) if gather_s > 0 else None,
        "gather_model_frac": (work["gather"][1] / gather_s / 1e9 / PEAK_HBM_GBS) if gather_s > 0 else None,
        "attention_exp_per_s": attention_exp_rate(wl, profile_tag(wl, head), B, prof),
        "phases": phase_rooflines(work, prof, wl.dtype == "bf16"),
        "kernels": kernels,
    }
    mfma = mfma_counter_rates(wl, tag, prof)
    if mfma:
        out["gemm_counter_tflops"] = mfma
    if wl.num_cat > 0 and not args.no_q8:
        out["gather_q8"] = time_gather_q8(db, work["gather_q8"][1], work["gather"][1])
    if args.graph:
        out["graph"] = time_graph_replays(step, args.steps, B)
    if cpu is not None:
        out["cpu_baseline"] = cpu
    print(json.dumps(out), flush=True)


def workload_description(wl, B: int, head) -> str:
    hot = ("%d multi-hot features (bags ~Poisson(%g) in [%d, %d])" % (wl.num_cat, wl.bag_mean, wl.bag_min, wl.bag_max)
           if wl.multi_hot else "%d single-hot features" % wl.num_cat)
    act = {"storage": "", "hilo": ", activations as bf16 hi + lo pairs",
           "f16": ", activations x_l and h held in f16 (bf16 weights and storage)"}[wl.act_mode]
    return ("%s: batch %d, %s (vocab %d, QR tables %dx%d, %s combine), %d dense, d=%d, %d Residual-DCN layers "
            "rank %d, attention %s%s%s" % (wl.name, B, hot, wl.vocab, wl.table_rows, wl.emb_dim, wl.combine,
                                          wl.num_dense, wl.d, wl.num_layers, wl.rank,
                                          "on" if wl.attention else "off",
                                          ", parallel plain branch" if wl.parallel else "", act)
            + (", Murmur-hashed ids (two QR pairs of 2^16 x 2^16 rows per feature)" if wl.hashed else "")
            + ("; head: %s%d x %s ReLU layers, logit, isotonic calibration (%d buckets), log loss"
               % ("gated " if head.gated else "", len(head.hidden),
                  "/".join(str(v) for v in sorted(set(head.hidden))), head.buckets) if head is not None else ""))


if __name__ == "__main__":
    main()
