"""The C-ABI library on a host without a GPU: it loads, exports every symbol
include/stage.h declares, validates arguments with the documented codes, and
reports a missing device instead of crashing (CPU only)."""

from __future__ import annotations

import os
import re

import numpy as np
import pytest
import torch

from paper_2606_18600_amd import stage as S
from paper_2606_18600_amd import synth
from paper_2606_18600_amd.harness import model_config

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _lib():
    if not os.path.exists(S.LIB_PATH):
        from paper_2606_18600_amd import build
        build.build(verbose=False)
    return S.load_library()


def header_functions():
    names = set()
    for f in os.listdir(os.path.join(ROOT, "include")):
        if f.endswith(".h"):
            src = open(os.path.join(ROOT, "include", f)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names |= set(re.findall(r"\b(stage_[a-z_]+)\s*\(", src))
    return names


def test_library_exports_every_declared_symbol():
    lib = _lib()
    declared = header_functions()
    assert {"stage_create", "stage_prefill", "stage_decode", "stage_step_mixed"} <= declared
    for name in sorted(declared):
        assert hasattr(lib, name), f"{name} declared in include/ but not exported"
    assert declared == set(S.EXPORTED)


CFG = model_config(synth.TINY, "bf16", max_position=4096)
FAKE_TABLE = 0x1000  # never dereferenced by host-side validation


def _b(q, c, mb=8, bt=FAKE_TABLE):
    return S.make_batch(q, c, bt, mb)


@pytest.mark.parametrize("case,code", [
    ("ok_prefill", S.STAGE_OK),
    ("ok_mixed", S.STAGE_OK),
    ("q_len_zero", S.STAGE_ERR_INVALID_ARG),
    ("decode_q_len_two", S.STAGE_ERR_INVALID_ARG),
    ("negative_ctx", S.STAGE_ERR_INVALID_ARG),
    ("null_table", S.STAGE_ERR_INVALID_ARG),
    ("table_too_small", S.STAGE_ERR_CAPACITY),
    ("too_many_tokens", S.STAGE_ERR_CAPACITY),
    ("too_many_seqs", S.STAGE_ERR_CAPACITY),
    ("past_max_position", S.STAGE_ERR_CAPACITY),
    ("empty", S.STAGE_OK),
])
def test_validate_step_codes(case, code):
    _lib()
    pf = dc = None
    mt, ms = 256, 8
    if case == "ok_prefill":
        pf = _b([17, 64], [0, 40])
    elif case == "ok_mixed":
        pf, dc = _b([16], [0]), _b([1, 1, 1], [0, 5, 127])
    elif case == "q_len_zero":
        pf = _b([3, 0], [0, 0])
    elif case == "decode_q_len_two":
        dc = S.make_batch([1, 2], [4, 4], FAKE_TABLE, 8)
    elif case == "negative_ctx":
        pf = _b([3], [-1])
    elif case == "null_table":
        pf = _b([3], [0], bt=0)
    elif case == "table_too_small":
        pf = _b([20], [100], mb=7)          # 120 tokens > 7 * 16
    elif case == "too_many_tokens":
        pf = _b([200, 57], [0, 0], mb=16)
    elif case == "too_many_seqs":
        dc = _b([1] * 9, [3] * 9)
    elif case == "past_max_position":
        pf = _b([2], [4095], mb=1024)
    elif case == "empty":
        pass
    got = S.stage_validate_step(CFG, mt, ms, pf, dc)
    assert got == code, S.stage_last_error()
    if code != S.STAGE_OK:
        assert S.stage_last_error()


@pytest.mark.parametrize("field,value,code", [
    ("head_dim", 96, S.STAGE_ERR_UNSUPPORTED),
    ("block_size", 32, S.STAGE_ERR_UNSUPPORTED),
    ("n_kv_heads", 3, S.STAGE_ERR_UNSUPPORTED),
    ("hidden", 200, S.STAGE_ERR_UNSUPPORTED),
    ("ffn", 0, S.STAGE_ERR_INVALID_ARG),
    ("dtype", 7, S.STAGE_ERR_UNSUPPORTED),
    ("rope_theta", -1.0, S.STAGE_ERR_INVALID_ARG),
])
def test_validate_config_codes(field, value, code):
    _lib()
    cfg = model_config(synth.TINY, "bf16")
    setattr(cfg, field, value)
    assert S.stage_validate_step(cfg, 16, 4, None, None) == code


@pytest.mark.skipif(torch.cuda.is_available(), reason="checks the no-device path")
def test_create_without_device_reports_device_error():
    _lib()
    ws = S.stage_layer_weights(*([0x1000] * 8))
    with pytest.raises(S.StageError) as e:
        S.stage_create(CFG, 0, 1, [ws], 0x2000, 16, 64, 4)
    assert e.value.code == S.STAGE_ERR_DEVICE


def test_create_rejects_bad_arguments_before_touching_a_device():
    _lib()
    ws = S.stage_layer_weights(*([0x1000] * 8))
    with pytest.raises(S.StageError) as e:
        S.stage_create(CFG, 3, 3, [ws], 0x2000, 16, 64, 4)       # empty layer range
    assert e.value.code == S.STAGE_ERR_INVALID_ARG
    bad = S.stage_layer_weights(*([0x1000] * 8))
    bad.w_down = None
    with pytest.raises(S.StageError) as e:
        S.stage_create(CFG, 0, 1, [bad], 0x2000, 16, 64, 4)
    assert e.value.code == S.STAGE_ERR_INVALID_ARG


def test_null_stage_calls_fail_cleanly():
    lib = _lib()
    assert lib.stage_prefill(None, None, None, None, None) == S.STAGE_ERR_INVALID_ARG
    assert lib.stage_destroy(None) == S.STAGE_OK
    assert lib.stage_workspace_bytes(None) == 0


@pytest.mark.parametrize("src,dst,nbytes", [
    (0, 0x2000, 64),            # NULL source
    (0x1000, 0, 64),            # NULL destination
    (0x1000, 0x2000, 40),       # size not a multiple of 16
    (0x1008, 0x2000, 64),       # misaligned source
    (0x1000, 0x1020, 64),       # overlapping buffers
])
def test_copy_probe_rejects_bad_arguments_on_the_host(src, dst, nbytes):
    lib = _lib()
    assert lib.stage_copy_probe(src, dst, nbytes, None) == S.STAGE_ERR_INVALID_ARG
    assert S.stage_last_error()


@pytest.mark.parametrize("vocab,src,dst,code", [
    (1024, 0, 0x2000, S.STAGE_ERR_INVALID_ARG),      # NULL source
    (1024, 0x1000, 0x1000, S.STAGE_ERR_INVALID_ARG),  # in place
    (0, 0x1000, 0x2000, S.STAGE_ERR_INVALID_ARG),     # empty vocabulary
    (1000, 0x1000, 0x2000, S.STAGE_ERR_UNSUPPORTED),  # bf16 vocab not a multiple of 128
])
def test_pack_lm_head_rejects_bad_arguments_on_the_host(vocab, src, dst, code):
    lib = _lib()
    cfg = model_config(synth.TINY, "bf16")
    assert lib.stage_pack_lm_head(cfg, vocab, src, dst, None) == code
    assert S.stage_last_error()


def test_lm_head_rejects_a_null_stage():
    lib = _lib()
    assert lib.stage_lm_head(None, 0x1000, 0x2000, 1024, 0x3000, 4, None, 4, 0x4000,
                             None) == S.STAGE_ERR_INVALID_ARG


def test_store_host_checks():
    """The store's argument checks need no device: empty and 2 GiB
    allocations are refused before anything is allocated; freeing or
    detaching NULL is a no-op."""
    lib = _lib()
    import ctypes
    p = ctypes.c_void_p()
    h = S.stage_ipc_handle()
    assert lib.stage_store_alloc(0, ctypes.byref(p), ctypes.byref(h)) == S.STAGE_ERR_INVALID_ARG
    assert lib.stage_store_alloc(1 << 31, ctypes.byref(p), ctypes.byref(h)) == \
        S.STAGE_ERR_CAPACITY
    assert "below" in S.stage_last_error()
    assert lib.stage_store_alloc(16, None, ctypes.byref(h)) == S.STAGE_ERR_INVALID_ARG
    assert lib.stage_store_attach(None, ctypes.byref(p)) == S.STAGE_ERR_INVALID_ARG
    assert lib.stage_store_free(None) == S.STAGE_OK
    assert lib.stage_store_detach(None) == S.STAGE_OK
    with pytest.raises(S.StageError):
        S.stage_store_attach(b"short")


def test_host_code_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    """The library's host code (stage.cpp, store.cpp, plan.cpp) built with
    g++ -fsanitize=address,undefined against a host-only stand-in of the HIP
    runtime, and driven by tests/host/stage_host_check.cpp: random valid and
    invalid steps on eight shapes in both dtypes (debug mode and op timing
    included), the allocation-free decode, the LM head and the store calls.
    Its launcher stubs read the step metadata back and check it (decode
    splits cover each token's keys exactly, prefill work items cover the
    rows once). Any sanitizer report or failed check fails the test."""
    import shutil
    import subprocess
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    src = os.path.join(ROOT, "paper_2606_18600_amd", "csrc")
    exe = str(tmp_path / "stage_host_check")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "tests", "host", "include"),
           os.path.join(ROOT, "tests", "host", "stage_host_check.cpp"),
           os.path.join(src, "stage.cpp"), os.path.join(src, "store.cpp"),
           os.path.join(src, "plan.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0 and "host check passed" in r.stdout, \
        (r.stdout[-2000:] + r.stderr[-4000:])
