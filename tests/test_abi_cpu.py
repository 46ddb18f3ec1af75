"""Host-side checks of the C ABI (no GPU): libcllm.so loads, exports every function that
include/cllm.h declares, and rejects bad arguments before touching the device."""
import ctypes
import os
import re
import struct

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cllm.h")


@pytest.fixture(scope="module")
def lib():
    from paper_2403_00835_amd import binding
    if not os.path.exists(binding.LIB_PATH):
        from paper_2403_00835_amd import build
        build.build()
    return binding.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cllm_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_paper_calls():
    names = declared_functions()
    for n in ["cllm_model_load", "cllm_prefill", "cllm_jacobi_step", "cllm_jacobi_decode"]:
        assert n in names


def test_library_exports_every_declared_function(lib):
    names = declared_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), n


def test_binding_names_match_header():
    from paper_2403_00835_amd import binding
    assert sorted(binding.EXPORTS) == declared_functions()


def test_status_strings(lib):
    for s in range(9):
        assert lib.cllm_status_string(s)
    assert lib.cllm_status_string(99) == b"unknown status"
    assert lib.cllm_last_error(None) == b"null context"


def test_null_arguments_rejected_without_device(lib):
    from paper_2403_00835_amd import binding
    h = ctypes.c_void_p()
    opts = binding.cllm_runtime_opts(64, 8, 8, 0, None)
    assert lib.cllm_model_create(None, ctypes.byref(opts), ctypes.byref(h)) == 1
    y = ctypes.c_int32()
    assert lib.cllm_prefill(None, 0, None, 0, ctypes.byref(y)) == 1
    a = ctypes.c_int32()
    assert lib.cllm_jacobi_step(None, 0, None, 1, None, ctypes.byref(a)) == 1
    assert lib.cllm_jacobi_decode(None, 0, None, 1, 1, 1, None, None, None) == 1
    assert lib.cllm_ar_decode(None, 0, None, 1, 1, None, None) == 1
    assert lib.cllm_model_load(None, ctypes.byref(opts), ctypes.byref(h)) == 1
    assert lib.cllm_model_load(b"/nonexistent/weights.bin", ctypes.byref(opts), ctypes.byref(h)) == 5
    assert lib.cllm_streamed_weight_bytes(None) == 0


def test_bad_config_rejected_before_device(lib):
    from paper_2403_00835_amd import binding
    h = ctypes.c_void_p()
    opts = binding.cllm_runtime_opts(64, 8, 8, 0, None)
    bad = binding.cllm_config(2, 64, 4, 15, 172, 256, 1e-6, 10000.0, 0)  # heads * head_dim != d
    assert lib.cllm_model_create(ctypes.byref(bad), ctypes.byref(opts), ctypes.byref(h)) == 1
    cfg = binding.cllm_config(2, 64, 4, 16, 172, 256, 1e-6, 10000.0, 0)
    too_big_block = binding.cllm_runtime_opts(64, 65, 8, 0, None)
    assert lib.cllm_model_create(ctypes.byref(cfg), ctypes.byref(too_big_block), ctypes.byref(h)) == 1
    for chunk in (-1, 4097):  # prefill chunk outside [0, 4096]
        bad_chunk = binding.cllm_runtime_opts(64, 8, 8, 0, None, 1, chunk)
        assert lib.cllm_model_create(ctypes.byref(cfg), ctypes.byref(bad_chunk), ctypes.byref(h)) == 1


def test_weight_file_header_layout(tmp_path):
    from paper_2403_00835_amd import binding, workload
    from paper_2403_00835_amd.configs import TINY
    ws = workload.make_weights(TINY)
    path = tmp_path / "w.bin"
    binding.write_weight_file(str(path), TINY, ws)
    raw = path.read_bytes()
    assert raw[:8] == b"CLLMWTS1"
    fields = struct.unpack("<i6i2fi", raw[8:48])
    assert fields[:7] == (1, 2, 64, 4, 16, 172, 256)
    assert abs(fields[7] - 1e-6) < 1e-12 and fields[8] == 10000.0 and fields[9] == 0
    assert len(raw) == 64 + sum(t.nbytes for t in ws)


def test_truncated_weight_file_rejected(lib, tmp_path):
    from paper_2403_00835_amd import binding
    h = ctypes.c_void_p()
    opts = binding.cllm_runtime_opts(64, 8, 8, 0, None)
    p = tmp_path / "bad.bin"
    p.write_bytes(b"NOTCLLM!" + b"\0" * 56)
    assert lib.cllm_model_load(str(p).encode(), ctypes.byref(opts), ctypes.byref(h)) == 6


def test_workspace_bytes_without_device(lib):
    # the size query needs no GPU; it grows with the row capacity and rejects what creation rejects
    from paper_2403_00835_amd import binding
    from paper_2403_00835_amd.configs import LLAMA7B, TINY
    a = binding.workspace_bytes(TINY, max_ctx=256, max_block=8, max_new=32)
    b = binding.workspace_bytes(TINY, max_ctx=256, max_block=8, max_new=32, max_batch=16)
    assert 0 < a < b and a % 256 == 0
    c = binding.workspace_bytes(LLAMA7B, max_ctx=704, max_block=16, max_new=256)
    assert c > 64 * 4096 * 4 * 5  # at least the 512-row activation planes
    with pytest.raises(binding.CllmError):
        binding.workspace_bytes(TINY, max_ctx=256, max_block=65, max_new=32)
