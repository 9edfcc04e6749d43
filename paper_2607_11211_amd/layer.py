"""ctypes binding of libfasttps.so (the C ABI in include/fasttps.h).

Argument marshalling only: every step of the decode layer runs in the HIP
kernels of the library. Device memory and streams come from PyTorch tensors
and streams. Importing this module loads the library and raises if it is
missing; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libfasttps.so")

OK = 0
ERR_INVALID_ARG = -1
ERR_UNSUPPORTED = -2
ERR_ALIGNMENT = -3
ERR_CACHE_FULL = -4
ERR_OOM = -5
ERR_HIP = -6
ERR_BAD_HANDLE = -7

DBG_QKV, DBG_ATTN, DBG_H1, DBG_MLP_A, DBG_FUSED_WAITS = 0, 1, 2, 3, 4
DBG_QK_ROPE, DBG_H, DBG_H2 = 5, 6, 7

GEMM_AUTO, GEMM_VECTOR, GEMM_MATRIX, GEMM_FUSED = 0, 1, 2, 3
MLP_SPLIT, MLP_FUSED = 0, 1
WEIGHTS_ROWS_AND_TILES, WEIGHTS_TILES = 0, 1

KV_FP8_E4M3 = 1
KV_INT8 = 2
KV_FORMATS = {"fp8_e4m3": KV_FP8_E4M3, "int8": KV_INT8}

EXPORTS = ("fasttps_layer_create", "fasttps_weights_pack", "fasttps_decode_step", "fasttps_debug_read",
           "fasttps_profile_begin", "fasttps_profile_end", "fasttps_kernel_name",
           "fasttps_unfused_enable", "fasttps_decode_step_unfused", "fasttps_set_attention_p_bf16",
           "fasttps_decode_step_kv8", "fasttps_set_gemm_path", "fasttps_set_debug", "fasttps_validate_step",
           "fasttps_set_mlp_path", "fasttps_decode_step_noalloc", "fasttps_set_weight_layout",
           "fasttps_weights_free", "fasttps_layer_destroy", "fasttps_status_string", "fasttps_last_error")
NUM_KERNELS = 7


class FastTPSError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: status {status} ({status_string(status)}): {detail}")
        self.status = status


class Config(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("intermediate", ctypes.c_int32), ("max_batch", ctypes.c_int32),
                ("max_seq", ctypes.c_int32), ("rope_base", ctypes.c_float), ("rms_eps", ctypes.c_float)]


WEIGHT_FIELDS = ("attn_norm", "w_q", "w_k", "w_v", "w_o", "mlp_norm", "w_gate", "w_up", "w_down")


class WeightsDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in WEIGHT_FIELDS]


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2607_11211_amd.build`")
    # One HIP runtime per process: torch carries its own libamdhip64 under the
    # same soname. Loaded first, it is the one this library binds to; loaded
    # after a ROCm copy, it would be a second runtime that finds no device.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    lib.fasttps_layer_create.argtypes = [ctypes.POINTER(Config), ctypes.POINTER(vp)]
    lib.fasttps_weights_pack.argtypes = [vp, ctypes.POINTER(WeightsDesc), vp, ctypes.POINTER(vp)]
    lib.fasttps_decode_step.argtypes = [vp, vp, vp, vp, i32, vp, vp, vp, vp]
    lib.fasttps_decode_step_unfused.argtypes = [vp, vp, vp, vp, i32, vp, vp, vp, vp]
    lib.fasttps_decode_step_noalloc.argtypes = [vp, vp, vp, vp, i32, vp, vp, vp, vp]
    fp = ctypes.POINTER(ctypes.c_float)
    lib.fasttps_decode_step_kv8.argtypes = [vp, vp, vp, vp, i32, i32, vp, vp, fp, fp, vp, vp]
    lib.fasttps_unfused_enable.argtypes = [vp]
    lib.fasttps_set_attention_p_bf16.argtypes = [vp, i32]
    lib.fasttps_set_gemm_path.argtypes = [vp, i32]
    lib.fasttps_set_debug.argtypes = [vp, i32]
    lib.fasttps_set_mlp_path.argtypes = [vp, i32]
    lib.fasttps_set_weight_layout.argtypes = [vp, i32]
    lib.fasttps_validate_step.argtypes = [ctypes.POINTER(Config), vp, ctypes.POINTER(i32), i32, vp, vp, vp, i32]
    lib.fasttps_debug_read.argtypes = [vp, i32, i32, vp, sz, vp]
    lib.fasttps_profile_begin.argtypes = [vp, i32]
    lib.fasttps_profile_end.argtypes = [vp, ctypes.POINTER(ctypes.c_float), i32, ctypes.POINTER(i32)]
    lib.fasttps_kernel_name.argtypes = [i32]
    lib.fasttps_kernel_name.restype = ctypes.c_char_p
    lib.fasttps_weights_free.argtypes = [vp]
    lib.fasttps_layer_destroy.argtypes = [vp]
    lib.fasttps_status_string.argtypes = [ctypes.c_int]
    lib.fasttps_status_string.restype = ctypes.c_char_p
    lib.fasttps_last_error.argtypes = []
    lib.fasttps_last_error.restype = ctypes.c_char_p
    for name in ("fasttps_layer_create", "fasttps_weights_pack", "fasttps_decode_step", "fasttps_debug_read",
                 "fasttps_profile_begin", "fasttps_profile_end", "fasttps_weights_free",
                 "fasttps_layer_destroy", "fasttps_unfused_enable", "fasttps_decode_step_unfused",
                 "fasttps_set_attention_p_bf16", "fasttps_decode_step_kv8", "fasttps_set_gemm_path",
                 "fasttps_set_debug", "fasttps_validate_step", "fasttps_decode_step_noalloc",
                 "fasttps_set_mlp_path", "fasttps_set_weight_layout"):
        getattr(lib, name).restype = ctypes.c_int
    return lib


LIB = _load()


def status_string(status: int) -> str:
    return LIB.fasttps_status_string(int(status)).decode()


def last_error() -> str:
    return LIB.fasttps_last_error().decode()


def _check(status: int, where: str) -> None:
    if status != OK:
        raise FastTPSError(status, where, last_error())


def make_config(cfg, max_batch: Optional[int] = None) -> Config:
    """C config from a shape record (``configs.LayerConfig``)."""
    return Config(cfg.hidden, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.intermediate,
                  cfg.batch if max_batch is None else max_batch, cfg.max_seq, float(cfg.rope_base),
                  float(cfg.rms_eps))


def validate_step(cfg, x_addr: int, pos, k_addr: int, v_addr: int, y_addr: int, cache_elem_bytes: int = 2,
                  max_batch: Optional[int] = None) -> int:
    """Status of a step's argument checks against a layer config (host only:
    addresses are examined, never dereferenced; no GPU needed)."""
    c = make_config(cfg, max_batch)
    p = np.ascontiguousarray(np.asarray(pos, dtype=np.int32))
    return int(LIB.fasttps_validate_step(ctypes.byref(c), x_addr or None,
                                         p.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), int(p.shape[0]),
                                         k_addr or None, v_addr or None, y_addr or None, int(cache_elem_bytes)))


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return stream.cuda_stream or None


class Weights:
    """Packed weights of one layer (owned by the library)."""

    def __init__(self, layer: "Layer", tensors: Dict[str, "object"], stream=None):
        desc = WeightsDesc(*[_ptr(tensors[n]) for n in WEIGHT_FIELDS])
        h = ctypes.c_void_p()
        _check(LIB.fasttps_weights_pack(layer.handle, ctypes.byref(desc), _stream_handle(stream),
                                        ctypes.byref(h)), "fasttps_weights_pack")
        self.handle = h

    def free(self) -> None:
        if self.handle:
            _check(LIB.fasttps_weights_free(self.handle), "fasttps_weights_free")
            self.handle = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


class Layer:
    """A decode-layer handle: config, scratch and RoPE table on the current device."""

    def __init__(self, cfg, max_batch: Optional[int] = None):
        self.cfg = cfg
        self.c = make_config(cfg, max_batch)
        h = ctypes.c_void_p()
        _check(LIB.fasttps_layer_create(ctypes.byref(self.c), ctypes.byref(h)), "fasttps_layer_create")
        self.handle = h
        self._h = h.value
        # host staging of the positions a step passes (read by the call itself)
        self._pos = (ctypes.c_int32 * 64)()
        self._pos_addr = ctypes.addressof(self._pos)

    def _stage_pos(self, pos):
        """Host address and length of pos (int32) for a step call: copied into
        the handle's staging array (the library reads it during the call, so
        one array serves every call); past 64 entries into a fresh array, for
        the library to refuse."""
        vals = pos.tolist() if isinstance(pos, np.ndarray) else list(pos)
        n = len(vals)
        if n > 64:
            self._pos_big = (ctypes.c_int32 * n)(*vals)
            return ctypes.addressof(self._pos_big), n
        buf = self._pos
        for i, v in enumerate(vals):
            buf[i] = v
        return self._pos_addr, n

    def pack(self, tensors: Dict[str, "object"], stream=None) -> Weights:
        return Weights(self, tensors, stream)

    def step(self, weights: Weights, x, pos, k_cache, v_cache, y, stream=None) -> None:
        """Enqueue one decode step. pos: host ints [batch]; tensors: torch device tensors.
        (Kept lean: on a 32-layer stack the host issues every layer's step.)"""
        pa, n = self._stage_pos(pos)
        st = LIB.fasttps_decode_step(self._h, weights.handle, x.data_ptr(), pa, n,
                                     k_cache.data_ptr(), v_cache.data_ptr(), y.data_ptr(),
                                     _stream_handle(stream))
        if st:
            _check(st, "fasttps_decode_step")

    def step_noalloc(self, weights: Weights, x, pos, k_cache, v_cache, y, stream=None) -> None:
        """Enqueue one decode step that allocates nothing (the library's static
        scratch array; vector-path kernels). Same contract as step."""
        pa, n = self._stage_pos(pos)
        _check(LIB.fasttps_decode_step_noalloc(self._h, weights.handle, _ptr(x), pa, n,
                                               _ptr(k_cache), _ptr(v_cache), _ptr(y), _stream_handle(stream)),
               "fasttps_decode_step_noalloc")

    def step_kv8(self, weights: Weights, fmt: str, x, pos, k_cache, v_cache, k_scale, v_scale, y,
                 stream=None) -> None:
        """Enqueue one decode step over an 8-bit cache (fmt "fp8_e4m3" or "int8").

        k_cache, v_cache: uint8 device tensors [batch, H_kv, N_max, d] of codes;
        k_scale, v_scale: host float sequences [H_kv], the per-KV-head scales.
        """
        if fmt not in KV_FORMATS:
            raise ValueError(f"unknown 8-bit KV format {fmt!r}")
        pa, n = self._stage_pos(pos)
        ks = np.ascontiguousarray(np.asarray(k_scale, dtype=np.float32))
        vs = np.ascontiguousarray(np.asarray(v_scale, dtype=np.float32))
        if ks.shape != (self.cfg.n_kv_heads,) or vs.shape != (self.cfg.n_kv_heads,):
            raise ValueError(f"scales must have shape ({self.cfg.n_kv_heads},)")
        fptr = ctypes.POINTER(ctypes.c_float)
        _check(LIB.fasttps_decode_step_kv8(self._h, weights.handle, _ptr(x), pa, n,
                                           KV_FORMATS[fmt], _ptr(k_cache), _ptr(v_cache),
                                           ks.ctypes.data_as(fptr), vs.ctypes.data_as(fptr), _ptr(y),
                                           _stream_handle(stream)),
               "fasttps_decode_step_kv8")

    def enable_unfused(self) -> None:
        """Allocate the op-by-op baseline's scratch (once per handle)."""
        _check(LIB.fasttps_unfused_enable(self.handle), "fasttps_unfused_enable")

    def step_unfused(self, weights: Weights, x, pos, k_cache, v_cache, y, stream=None) -> None:
        """Enqueue one step of the op-by-op baseline (same contract as step)."""
        pa, n = self._stage_pos(pos)
        _check(LIB.fasttps_decode_step_unfused(self._h, weights.handle, _ptr(x), pa, n,
                                               _ptr(k_cache), _ptr(v_cache), _ptr(y), _stream_handle(stream)),
               "fasttps_decode_step_unfused")

    def set_gemm_path(self, path: int) -> None:
        """Projection kernels: GEMM_AUTO, GEMM_VECTOR (GEMVs), GEMM_MATRIX (MFMA; max_batch > 1)
        or GEMM_FUSED (one sequence, the whole step as one persistent kernel)."""
        _check(LIB.fasttps_set_gemm_path(self.handle, int(path)), "fasttps_set_gemm_path")

    def fused_wait_errors(self) -> int:
        """Bounded waits of the fused kernel that ran out since the layer was created."""
        import torch
        t = torch.zeros(1, dtype=torch.int32, device="cuda")
        _check(LIB.fasttps_debug_read(self.handle, DBG_FUSED_WAITS, 1, _ptr(t), 4, _stream_handle(None)),
               "fasttps_debug_read")
        torch.cuda.synchronize()
        return int(t.item())

    def set_mlp_path(self, path: int) -> None:
        """MLP_SPLIT (gate/up stores h^sm, down reads it) or MLP_FUSED (h^sm kept on chip;
        weights must be packed after selecting it)."""
        _check(LIB.fasttps_set_mlp_path(self.handle, int(path)), "fasttps_set_mlp_path")

    def set_weight_layout(self, layout: int) -> None:
        """WEIGHTS_ROWS_AND_TILES (default) or WEIGHTS_TILES (the MFMA tile order only; every
        step with such weights runs the matrix path); applies to weights packed afterwards."""
        _check(LIB.fasttps_set_weight_layout(self.handle, int(layout)), "fasttps_set_weight_layout")

    def set_debug(self, enable: bool) -> None:
        """Test hook: later steps also write q, k after RoPE and the two normalized activations."""
        _check(LIB.fasttps_set_debug(self.handle, 1 if enable else 0), "fasttps_set_debug")

    def set_attention_p_bf16(self, enable: bool) -> None:
        """Accuracy study only: round the softmax weights to bf16 before PV."""
        _check(LIB.fasttps_set_attention_p_bf16(self.handle, 1 if enable else 0), "fasttps_set_attention_p_bf16")

    def debug_read(self, which: int, batch: int, dst, stream=None) -> None:
        _check(LIB.fasttps_debug_read(self.handle, int(which), int(batch), _ptr(dst),
                                      int(dst.numel() * dst.element_size()), _stream_handle(stream)),
               "fasttps_debug_read")

    def profile_begin(self, max_steps: int) -> None:
        _check(LIB.fasttps_profile_begin(self.handle, int(max_steps)), "fasttps_profile_begin")

    def profile_end(self, max_steps: int) -> np.ndarray:
        """Per-kernel milliseconds [n_steps, NUM_KERNELS] of the recorded steps."""
        ms = np.zeros((max_steps, NUM_KERNELS), dtype=np.float32)
        n = ctypes.c_int32(0)
        _check(LIB.fasttps_profile_end(self.handle, ms.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                                       int(max_steps), ctypes.byref(n)), "fasttps_profile_end")
        return ms[: n.value]

    def destroy(self) -> None:
        if self.handle:
            _check(LIB.fasttps_layer_destroy(self.handle), "fasttps_layer_destroy")
            self.handle = None
            self._h = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def kernel_names():
    return [LIB.fasttps_kernel_name(k).decode() for k in range(NUM_KERNELS)]


def to_device(bits: np.ndarray, device="cuda"):
    """Upload bf16 bit patterns (uint16) as an int16 device tensor (same bytes)."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(device)


def from_device(t) -> np.ndarray:
    """Download an int16/bf16 device tensor as uint16 bit patterns."""
    import torch
    if t.dtype == torch.bfloat16:
        t = t.view(torch.int16)
    return t.cpu().numpy().view(np.uint16)
