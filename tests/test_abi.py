"""The C ABI library loads, exports everything include/rdcn.h declares, and
rejects bad arguments on the host before any GPU work (CPU-only tests)."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2402_06859_amd import rdcn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rdcn.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\**\s+\**(\w+)\s*\(", src, flags=re.M)))


def test_header_declares_binding_exports():
    assert declared_functions() == sorted(rdcn.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = rdcn.load()
    for name in declared_functions():
        assert hasattr(L, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", rdcn.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (\w+)", out))
    assert set(declared_functions()) <= exported


def test_struct_layout_matches_c(tmp_path):
    prog = tmp_path / "layout.c"
    prog.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "rdcn.h"\n'
                    'int main(void){printf("%zu %zu %zu %zu %zu\\n", sizeof(rdcn_config), offsetof(rdcn_config, vocab),'
                    ' offsetof(rdcn_config, temperature), sizeof(rdcn_weights), offsetof(rdcn_weights, bias));'
                    'return 0;}\n')
    exe = tmp_path / "layout"
    subprocess.check_call(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), str(prog), "-o", str(exe)])
    vals = [int(v) for v in subprocess.check_output([str(exe)]).split()]
    C, W = rdcn.RdcnConfig, rdcn.RdcnWeights
    assert vals == [ctypes.sizeof(C), C.vocab.offset, C.temperature.offset, ctypes.sizeof(W), W.bias.offset]


def test_status_strings():
    for s in range(8):
        assert rdcn.status_string(s) != "unknown status"
    assert rdcn.status_string(99) == "unknown status"


def good():
    return rdcn.make_config(64, 4, 16, 32, 8, 2, 25, 25, 600, "sum", False, "i64", "bf16", 1.0, 1.0, 1.0)


@pytest.mark.parametrize("field,value,expect", [
    ("num_layers", 0, rdcn.RDCN_ERR_ARG), ("num_layers", 17, rdcn.RDCN_ERR_ARG), ("rank", 0, rdcn.RDCN_ERR_ARG),
    ("emb_dim", 0, rdcn.RDCN_ERR_ARG), ("num_cat", -1, rdcn.RDCN_ERR_ARG), ("batch_max", -1, rdcn.RDCN_ERR_ARG),
    ("combine", 7, rdcn.RDCN_ERR_ARG), ("dtype", 3, rdcn.RDCN_ERR_ARG), ("id_type", 2, rdcn.RDCN_ERR_ARG),
    ("temperature", 0.0, rdcn.RDCN_ERR_ARG), ("temperature", -1.0, rdcn.RDCN_ERR_ARG), ("vocab", 0, rdcn.RDCN_ERR_ARG),
    ("activation_mode", 3, rdcn.RDCN_ERR_ARG), ("activation_mode", -1, rdcn.RDCN_ERR_ARG), ("multi_hot", 2, rdcn.RDCN_ERR_ARG),
    ("vocab", 626, rdcn.RDCN_ERR_SHAPE),                      # 25 * 25 < 626: ids would not fit the tables
    ("emb_dim", 12, rdcn.RDCN_ERR_UNSUPPORTED), ("num_dense", 4, rdcn.RDCN_ERR_UNSUPPORTED),
    ("rank", 12, rdcn.RDCN_ERR_UNSUPPORTED), ("emb_dim", 264, rdcn.RDCN_ERR_UNSUPPORTED),
])
def test_create_rejects_bad_config_before_hip(field, value, expect):
    c = good()
    setattr(c, field, value)
    h = ctypes.c_void_p()
    assert rdcn.load().rdcn_create(ctypes.byref(c), ctypes.byref(h)) == expect
    assert not h.value


@pytest.mark.parametrize("mode", [1, 2])
def test_activation_modes_need_bf16(mode):
    c = good()
    c.dtype, c.emb_dim, c.num_dense, c.rank, c.activation_mode = rdcn.F32, 16, 32, 8, mode
    h = ctypes.c_void_p()
    assert rdcn.load().rdcn_create(ctypes.byref(c), ctypes.byref(h)) == rdcn.RDCN_ERR_UNSUPPORTED


def test_side_stream_switch_rejects_null_handle():
    assert rdcn.load().rdcn_set_side_stream(None, 0) == rdcn.RDCN_ERR_ARG
    assert rdcn.load().rdcn_set_side_stream(None, 1) == rdcn.RDCN_ERR_ARG


def test_create_null_arguments():
    L = rdcn.load()
    h = ctypes.c_void_p()
    assert L.rdcn_create(None, ctypes.byref(h)) == rdcn.RDCN_ERR_ARG
    assert L.rdcn_create(ctypes.byref(good()), None) == rdcn.RDCN_ERR_ARG


def test_entry_points_reject_null_handle():
    L = rdcn.load()
    sz = ctypes.c_size_t()
    i = ctypes.c_int64()
    w = rdcn.RdcnWeights()
    assert L.rdcn_dim(None, ctypes.byref(i)) == rdcn.RDCN_ERR_ARG
    assert L.rdcn_workspace_bytes(None, 1, ctypes.byref(sz), ctypes.byref(sz)) == rdcn.RDCN_ERR_ARG
    assert L.qr_embed_gather(None, 1, None, None, None, None, None, None, None) == rdcn.RDCN_ERR_ARG
    assert L.qr_embed_backward_workspace(None, 1, 1, ctypes.byref(sz)) == rdcn.RDCN_ERR_ARG
    assert L.qr_embed_backward(None, 1, 1, None, None, None, None, None, None, None, None, 0, None) == rdcn.RDCN_ERR_ARG
    assert L.rdcn_forward(None, 1, None, ctypes.byref(w), None, None, None, None) == rdcn.RDCN_ERR_ARG
    assert L.rdcn_backward(None, 1, None, ctypes.byref(w), None, None, None, ctypes.byref(w), None,
                           None) == rdcn.RDCN_ERR_ARG
    assert L.rdcn_check_device_errors(None, None) == rdcn.RDCN_ERR_ARG
    assert L.rdcn_destroy(None) == rdcn.RDCN_OK


def test_quantization_entry_points_reject_null_handle():
    L = rdcn.load()
    assert L.qr_quantize_tables(None, 4, None, None, None, None) == rdcn.RDCN_ERR_ARG
    assert L.qr_embed_gather_q8(None, 4, None, None, None, None, None, None, None, None, None) == rdcn.RDCN_ERR_ARG


def test_parallel_branch_validation():
    L = rdcn.load()
    h = ctypes.c_void_p()
    c = good()
    c.parallel_branch = 2
    assert L.rdcn_create(ctypes.byref(c), ctypes.byref(h)) == rdcn.RDCN_ERR_ARG
    c = good()
    c.parallel_branch, c.attn_alpha = 1, 0.0
    assert L.rdcn_create(ctypes.byref(c), ctypes.byref(h)) == rdcn.RDCN_ERR_ARG
    c = good()
    for mode in (1, 2):
        c.parallel_branch, c.activation_mode = 1, mode
        assert L.rdcn_create(ctypes.byref(c), ctypes.byref(h)) == rdcn.RDCN_ERR_UNSUPPORTED


def test_hashed_front_end_validation():
    L = rdcn.load()
    h = ctypes.c_void_p()
    c = good()
    c.hashed = 1  # vocab must be 0
    assert L.rdcn_create(ctypes.byref(c), ctypes.byref(h)) == rdcn.RDCN_ERR_ARG
    c.vocab = 0   # 25 * 25 rows do not cover a 32-bit hash half
    assert L.rdcn_create(ctypes.byref(c), ctypes.byref(h)) == rdcn.RDCN_ERR_SHAPE
    c = good()
    c.hashed = 2
    assert L.rdcn_create(ctypes.byref(c), ctypes.byref(h)) == rdcn.RDCN_ERR_ARG
    c = good()
    c.reserved2 = 1
    assert L.rdcn_create(ctypes.byref(c), ctypes.byref(h)) == rdcn.RDCN_ERR_ARG


def test_head_struct_layout_matches_c(tmp_path):
    prog = tmp_path / "hlayout.c"
    prog.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "rdcn.h"\n'
                    'int main(void){printf("%zu %zu %zu %zu %zu %zu\\n", sizeof(rdcn_head_config),'
                    ' offsetof(rdcn_head_config, gated), offsetof(rdcn_head_config, bucket_step),'
                    ' sizeof(rdcn_head_weights), offsetof(rdcn_head_weights, w_out), offsetof(rdcn_head_weights, cal_b));'
                    'return 0;}\n')
    exe = tmp_path / "hlayout"
    subprocess.check_call(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), str(prog), "-o", str(exe)])
    vals = [int(v) for v in subprocess.check_output([str(exe)]).split()]
    C, W = rdcn.RdcnHeadConfig, rdcn.RdcnHeadWeights
    assert vals == [ctypes.sizeof(C), C.gated.offset, C.bucket_step.offset, ctypes.sizeof(W), W.w_out.offset,
                    W.cal_b.offset]
    assert len(rdcn.KERNELS) == 27  # RDCN_KERNEL_COUNT: rdcn_profile_stop writes that many entries


def test_head_calls_reject_null_handle():
    L = rdcn.load()
    cfg = rdcn.make_head_config([16], True, 4, -1.0, 0.5)
    s, t = ctypes.c_size_t(), ctypes.c_size_t()
    w = rdcn.RdcnHeadWeights()
    assert L.rdcn_head_configure(None, ctypes.byref(cfg)) == rdcn.RDCN_ERR_ARG
    assert L.rdcn_head_workspace_bytes(None, 4, ctypes.byref(s), ctypes.byref(t)) == rdcn.RDCN_ERR_ARG
    assert L.rdcn_head_forward(None, 4, None, None, ctypes.byref(w), None, None, None, None) == rdcn.RDCN_ERR_ARG
    assert L.rdcn_head_logloss(None, 4, None, None, 1.0, None, None, None) == rdcn.RDCN_ERR_ARG
    assert L.rdcn_head_backward(None, 4, None, None, ctypes.byref(w), None, None, None, None, ctypes.byref(w), None,
                                None) == rdcn.RDCN_ERR_ARG
