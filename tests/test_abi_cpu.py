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
    f.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                  ctypes.c_void_p, ctypes.POINTER(ctypes.c_float)]
    ms = ctypes.c_float()
    a = ctypes.c_void_p(64)
    assert f(None, 16, a, 1, 1, 0, None, ctypes.byref(ms)) == -1   # null source
    assert f(a, 24, a, 1, 1, 0, None, ctypes.byref(ms)) == -1      # not a multiple of 16
    assert f(a, 16, a, 1, 3, 0, None, ctypes.byref(ms)) == -1      # unroll 3
    assert f(a, 16, a, 0, 1, 0, None, ctypes.byref(ms)) == -1      # no blocks
    assert f(a, 16, a, 1, 1, 2, None, ctypes.byref(ms)) == -1      # unknown load flavour


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


# ---- the step's argument checks, on the host (fasttps_validate_step) -------
# Fake device addresses: only their values are examined (alignment, overlap),
# nothing is dereferenced. Tiny layer: D 256, H_kv 4, N_max 256, d 64, so one
# sequence's bf16 cache is 4 * 256 * 64 * 2 = 128 KiB.
_CACHE = 4 * 256 * 64 * 2


def _shape(**kw):
    from paper_2607_11211_amd import configs
    import dataclasses
    return dataclasses.replace(configs.get("tiny"), **kw)


def _addrs(batch=1, elem=2):
    """x, k, v, y at disjoint 256-byte-aligned fake addresses."""
    cache = batch * _CACHE // 2 * elem
    x = 1 << 32
    k = x + (1 << 24)
    v = k + cache + 256
    y = v + cache + 256
    return x, k, v, y


def test_validate_step_accepts_a_good_step(L):
    x, k, v, y = _addrs()
    assert L.validate_step(_shape(), x, [128], k, v, y) == L.OK
    assert L.validate_step(_shape(), x, [0], k, v, y) == L.OK
    assert L.validate_step(_shape(), x, [255], k, v, y) == L.OK     # the last slot: N_r = 1


@pytest.mark.parametrize("pos", [[256], [300], [-1], [2 ** 31 - 1]])
def test_validate_step_cache_full(L, pos):
    x, k, v, y = _addrs()
    assert L.validate_step(_shape(), x, pos, k, v, y) == L.ERR_CACHE_FULL
    assert "pos[0]" in L.last_error()


def test_validate_step_cache_full_in_a_batch(L):
    x, k, v, y = _addrs(batch=3)
    cfg = _shape(batch=3, pos=(1, 2, 3))
    assert L.validate_step(cfg, x, [10, 255, 20], k, v, y) == L.OK
    assert L.validate_step(cfg, x, [10, 256, 20], k, v, y) == L.ERR_CACHE_FULL
    assert "pos[1]" in L.last_error()


@pytest.mark.parametrize("which", range(4))
def test_validate_step_alignment(L, which):
    a = list(_addrs())
    a[which] += 8
    x, k, v, y = a
    assert L.validate_step(_shape(), x, [5], k, v, y) == L.ERR_ALIGNMENT


@pytest.mark.parametrize("which", range(4))
def test_validate_step_null_pointers(L, which):
    a = list(_addrs())
    a[which] = 0
    x, k, v, y = a
    assert L.validate_step(_shape(), x, [5], k, v, y) == L.ERR_INVALID_ARG


def test_validate_step_batch_range(L):
    x, k, v, y = _addrs(batch=4)
    cfg = _shape(batch=2, pos=(1, 2))
    assert L.validate_step(cfg, x, [1, 2], k, v, y) == L.OK
    assert L.validate_step(cfg, x, [1, 2, 3], k, v, y) == L.ERR_INVALID_ARG   # batch 3 > max_batch 2
    assert "batch" in L.last_error()
    assert L.validate_step(cfg, x, [], k, v, y) == L.ERR_INVALID_ARG           # batch 0
    assert L.validate_step(cfg, x, [1, 2, 3, 4], k, v, y, max_batch=4) == L.OK


def test_validate_step_overlaps(L):
    x, k, v, y = _addrs()
    cfg = _shape()
    assert L.validate_step(cfg, x, [5], k, v, x) == L.ERR_INVALID_ARG            # y is x
    assert L.validate_step(cfg, x, [5], k, v, x + 256) == L.ERR_INVALID_ARG      # y inside x (512 B)
    assert L.validate_step(cfg, x, [5], k, v, x + 512) == L.OK                   # y right after x
    assert L.validate_step(cfg, x, [5], k, v, k + _CACHE - 256) == L.ERR_INVALID_ARG  # y in the K cache
    assert L.validate_step(cfg, x, [5], k, v, v) == L.ERR_INVALID_ARG            # y in the V cache
    assert L.validate_step(cfg, x, [5], k, k + _CACHE - 16, y) == L.ERR_INVALID_ARG  # caches overlap
    assert "overlap" in L.last_error()
    assert L.validate_step(cfg, x, [5], k, k + _CACHE, y) == L.OK                # caches adjacent


def test_validate_step_8bit_cache_extent(L):
    """An 8-bit cache is one byte per element: V may start half a bf16 cache after K."""
    x, k, v, y = _addrs(elem=1)
    cfg = _shape()
    assert L.validate_step(cfg, x, [5], k, k + _CACHE // 2, y, cache_elem_bytes=1) == L.OK
    assert L.validate_step(cfg, x, [5], k, k + _CACHE // 2, y, cache_elem_bytes=2) == L.ERR_INVALID_ARG
    assert L.validate_step(cfg, x, [5], k, v, y, cache_elem_bytes=3) == L.ERR_INVALID_ARG


def test_validate_step_checks_the_config(L):
    x, k, v, y = _addrs()
    assert L.validate_step(_shape(head_dim=80), x, [5], k, v, y) == L.ERR_UNSUPPORTED
    assert L.LIB.fasttps_validate_step(None, x, (ctypes.c_int32 * 1)(0), 1, k, v, y, 2) == L.ERR_INVALID_ARG


def test_debug_hooks_reject_bad_handles(L):
    assert L.LIB.fasttps_set_debug(None, 1) == L.ERR_BAD_HANDLE
    for which in (L.DBG_QK_ROPE, L.DBG_H, L.DBG_H2):
        assert L.LIB.fasttps_debug_read(None, which, 1, None, 0, None) == L.ERR_BAD_HANDLE
