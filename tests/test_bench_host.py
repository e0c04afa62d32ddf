"""Host logic of bench.py (no GPU): the one-GPU guard, the algorithmic work model,
the roofline bound selection, and the lookup of counter records by workload tag and
source hash."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2402_06859_amd.synth import HEADS, WORKLOADS  # noqa: E402


def test_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)


def test_work_model_by_hand_on_tiny():
    """Flops of the products and bytes of the gather, written out from the shapes."""
    wl = WORKLOADS["tiny"]
    B, d, r, F, D, Nd = wl.batch, wl.d, wl.rank, wl.num_cat, wl.emb_dim, wl.num_dense
    w = bench.kernel_work(wl, B)
    n = wl.n_proj
    assert w["fwd_down_gemm"][0] == 2.0 * B * n * r * d
    assert w["fwd_up_gemm"][0] == 2.0 * B * d * r
    assert w["bwd_gw_gemm"][0] == 2.0 * n * r * d * B
    assert w["bwd_gx_gemm"][0] == 2.0 * B * d * n * r
    eb = 4  # float storage
    # ids (8 bytes each), both table rows of every id, the embedding columns of x0, dense in and out
    assert w["gather"][1] == B * (F * 8 + 2 * F * D * eb + F * D * eb + 2 * Nd * eb)


def test_work_model_large_products():
    wl = WORKLOADS["large"]
    w = bench.kernel_work(wl, wl.batch)
    assert w["fwd_down_gemm"][0] == pytest.approx(2.139e12, rel=1e-3)   # 2 * 32768 * 3072 * 10624
    assert w["fwd_up_gemm"][0] == pytest.approx(7.13e11, rel=1e-3)
    # one exponential per (query, key) pair, carried as 7 FMA-equivalent flops per pair
    assert w["fwd_attention"][2] / 7.0 == pytest.approx(wl.batch * wl.rank * wl.rank)


def test_work_model_attention_bytes():
    """Bytes of the attention kernels written out from what they move per sample: the
    forward reads [v|q|k] (float) and writes h (bf16, plus its f16 copy when the
    activations are held in f16) and four float statistics per row (o, Z, W1, W2); the
    backward reads [v|q|k], the float gh and the statistics and writes [gv|gq|gk]."""
    wl = WORKLOADS["large"]  # f16 activations
    B, r = wl.batch, wl.rank
    w = bench.kernel_work(wl, B)
    assert w["fwd_attention"][1] == B * (3 * r * 4 + 2 * r * 2 + 4 * r * 4)
    assert w["bwd_attention"][1] == B * (3 * r * 4 + r * 4 + 4 * r * 4 + 3 * r * 2)
    # up: h, U, bias, x0, x_l in; t, x_{l+1} (f16) and its bf16 copy out
    d = wl.d
    assert w["fwd_up_gemm"][1] == B * r * 2 + d * r * 2 + d * 2 + B * d * 2 * 5
    small = WORKLOADS["small"]  # bf16 activations: one h plane
    ws = bench.kernel_work(small, small.batch)
    assert ws["fwd_attention"][1] == small.batch * (3 * small.rank * 4 + small.rank * 2 + 4 * small.rank * 4)


def test_roofline_bound_selection():
    # attention of a bf16 model: exponential-bound, reported in exponentials per second
    r = bench.roofline_for("fwd_attention", (0.0, 1e9, 7.0e12), 1e-3, True)
    assert r["bound"] == "exp" and r["unit"] == "Texp/s"
    assert r["achieved"] == pytest.approx(1e12 / 1e-3 / 1e12)
    # a product whose flops take longer at peak than its bytes: matrix-core-bound
    r = bench.roofline_for("fwd_down_gemm", (2.5e12, 1e9, 0.0), 2e-3, True)
    assert r["bound"] == "mfma" and r["peak"] == bench.PEAK_BF16_TFLOPS
    # a short product with a heavy epilogue: HBM-bound
    r = bench.roofline_for("fwd_up_gemm", (1e9, 8e9, 0.0), 2e-3, True)
    assert r["bound"] == "hbm" and r["achieved"] == pytest.approx(8e9 / 2e-3 / 1e9)


def test_profile_tags():
    wl = WORKLOADS["small"]
    assert bench.profile_tag(wl) == "small"
    assert bench.profile_tag(wl.with_(hashed=True, table_rows=1 << 16)) == "small+hashed"
    assert bench.profile_tag(wl.with_(parallel=True)) == "small+parallel"
    assert bench.profile_tag(WORKLOADS["feed"], HEADS["lmlp"]) == "feed+lmlp"


def test_counter_records_follow_the_sources(tmp_path, monkeypatch):
    """A record is used only for its kernel, workload tag and the SHA-256 of the kernel's
    current sources; any other hash reads as no record."""
    sha = bench.sources_sha256("gather")
    prof = tmp_path / "profiles"
    prof.mkdir()
    good = {"kernel": "gather", "workload": "small", "sha256": sha, "bytes_per_launch": 1234}
    stale = dict(good, workload="feed", sha256="0" * 64)
    (prof / "x_counters.md").write_text("notes\ntraffic: %s\ntraffic: %s\n" % (json.dumps(good), json.dumps(stale)))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "sources_sha256", lambda k: sha)
    assert bench.measured_traffic("gather", "small") == 1234
    assert bench.measured_traffic("gather", "feed") is None
    assert bench.measured_traffic("fwd_attention", "small") is None
    assert bench.counter_record("traffic", "gather", "small")["bytes_per_launch"] == 1234
