"""The C-ABI library on the CPU: it loads, exports what the header declares, and
rejects bad arguments before any HIP call (no GPU needed)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fasttps.h")


@pytest.fixture(scope="module")
def L():
    from paper_2607_11211_amd import build
    if not os.path.exists(build.LIB):
        build.build(verbose=False)
    import paper_2607_11211_amd.layer as layer
    return layer


def declared_functions():
    text = open(HEADER).read()
    return re.findall(r"FASTTPS_API\s+[\w\s\*]+?\b(fasttps_\w+)\s*\(", text)


def test_header_declares_the_abi():
    names = declared_functions()
    for n in ("fasttps_layer_create", "fasttps_weights_pack", "fasttps_decode_step", "fasttps_weights_free",
              "fasttps_layer_destroy", "fasttps_status_string", "fasttps_last_error", "fasttps_debug_read",
              "fasttps_profile_begin", "fasttps_profile_end", "fasttps_kernel_name"):
        assert n in names


def test_library_exports_every_declared_symbol(L):
    for name in declared_functions():
        assert hasattr(L.LIB, name), name
    assert set(declared_functions()) == set(L.EXPORTS)


def test_unfused_entry_points_reject_bad_handles(L):
    assert L.LIB.fasttps_unfused_enable(None) == L.ERR_BAD_HANDLE
    p = (ctypes.c_int32 * 1)(0)
    assert L.LIB.fasttps_decode_step_unfused(None, None, None, p, 1, None, None, None, None) == L.ERR_BAD_HANDLE


def test_gemm_path_hook_rejects_bad_handles(L):
    for path in (L.GEMM_AUTO, L.GEMM_VECTOR, L.GEMM_MATRIX, 7):
        assert L.LIB.fasttps_set_gemm_path(None, path) == L.ERR_BAD_HANDLE


def test_kv8_entry_point_rejects_bad_format_and_handles(L):
    p = (ctypes.c_int32 * 1)(0)
    sc = (ctypes.c_float * 1)(1.0)
    f = L.LIB.fasttps_decode_step_kv8
    for fmt in (0, 3, -1):
        assert f(None, None, None, p, 1, fmt, None, None, sc, sc, None, None) == L.ERR_INVALID_ARG
        assert "format" in L.last_error()
    for fmt in (L.KV_FP8_E4M3, L.KV_INT8):
        assert f(None, None, None, p, 1, fmt, None, None, sc, sc, None, None) == L.ERR_BAD_HANDLE


def test_probe_library_exports_its_header():
    """The measurement aid (stream-read probe) is a library of its own with
    its own header; it rejects bad arguments before touching the GPU."""
    from paper_2607_11211_amd import build
    if not os.path.exists(build.PROBE_LIB):
        build.build(verbose=False)
    text = open(os.path.join(ROOT, "include", "fasttps_probe.h")).read()
    names = re.findall(r"FASTTPS_PROBE_API\s+[\w\s\*]+?\b(fasttps_\w+)\s*\(", text)
    assert names == ["fasttps_probe_stream_read"]
    lib = ctypes.CDLL(build.PROBE_LIB)
    f = lib.fasttps_probe_stream_read
    f.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                  ctypes.POINTER(ctypes.c_float)]
    ms = ctypes.c_float()
    assert f(None, 16, ctypes.c_void_p(64), 1, 1, None, ctypes.byref(ms)) == -1      # null source
    assert f(ctypes.c_void_p(64), 24, ctypes.c_void_p(64), 1, 1, None, ctypes.byref(ms)) == -1  # not 16-multiple
    assert f(ctypes.c_void_p(64), 16, ctypes.c_void_p(64), 1, 3, None, ctypes.byref(ms)) == -1  # unroll 3
    assert f(ctypes.c_void_p(64), 16, ctypes.c_void_p(64), 0, 1, None, ctypes.byref(ms)) == -1  # no blocks


def test_status_strings(L):
    seen = set()
    for code in (0, -1, -2, -3, -4, -5, -6, -7):
        s = L.status_string(code)
        assert s and s != "unknown status"
        seen.add(s)
    assert len(seen) == 8
    assert L.status_string(-99) == "unknown status"


def _cfg(L, **kw):
    base = dict(hidden=256, n_heads=4, n_kv_heads=4, head_dim=64, intermediate=688, max_batch=1,
                max_seq=256, rope_base=10000.0, rms_eps=1e-5)
    base.update(kw)
    return L.Config(**base)


@pytest.mark.parametrize("kw,code", [
    (dict(head_dim=80), -2),
    (dict(hidden=100), -2),
    (dict(hidden=16384), -2),
    (dict(n_heads=6, n_kv_heads=2), -2),
    (dict(n_heads=6, n_kv_heads=4), -2),
    (dict(intermediate=689), -2),
    (dict(intermediate=32776), -2),
    (dict(rms_eps=0.0), -1),
    (dict(rope_base=float("nan")), -1),
    (dict(max_batch=65), -1),
    (dict(max_batch=0), -1),
    (dict(max_seq=0), -1),
    (dict(hidden=-8), -1),
])
def test_create_rejects_bad_config(L, kw, code):
    c = _cfg(L, **kw)
    h = ctypes.c_void_p()
    assert L.LIB.fasttps_layer_create(ctypes.byref(c), ctypes.byref(h)) == code
    assert not h.value
    assert L.last_error()


def test_create_null_arguments(L):
    h = ctypes.c_void_p()
    assert L.LIB.fasttps_layer_create(None, ctypes.byref(h)) == L.ERR_INVALID_ARG
    c = _cfg(L)
    assert L.LIB.fasttps_layer_create(ctypes.byref(c), None) == L.ERR_INVALID_ARG


def test_null_handles_are_rejected(L):
    assert L.LIB.fasttps_layer_destroy(None) == L.ERR_BAD_HANDLE
    assert L.LIB.fasttps_weights_free(None) == L.ERR_BAD_HANDLE
    assert L.LIB.fasttps_debug_read(None, 0, 1, None, 0, None) == L.ERR_BAD_HANDLE
    pos = (ctypes.c_int32 * 1)(0)
    assert L.LIB.fasttps_decode_step(None, None, None, pos, 1, None, None, None, None) == L.ERR_BAD_HANDLE
    h = ctypes.c_void_p()
    assert L.LIB.fasttps_weights_pack(None, None, None, ctypes.byref(h)) == L.ERR_BAD_HANDLE
    assert "handle" in L.last_error()


def test_create_without_gpu_fails_cleanly(L):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    c = _cfg(L)
    h = ctypes.c_void_p()
    assert L.LIB.fasttps_layer_create(ctypes.byref(c), ctypes.byref(h)) == L.ERR_HIP
    assert not h.value
