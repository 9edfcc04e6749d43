"""Seeded synthetic inputs for one decode step (shared by the oracle tests and the GPU path).

Recipe (the same bits feed the oracle and the library):
  * projection weights ~ N(0, 0.02), RMSNorm gains ~ 1 + 0.1 N(0, 1),
    token x ~ N(0, 1), cache entries [0, pos_b) ~ N(0, 1);
  * every value is drawn as float32 and rounded to bfloat16 (round to nearest,
    ties to even) once, here, so both sides start from identical bits;
  * cache slots [pos_b, max_seq) of every (sequence, kv head) hold quiet-NaN
    sentinels (0x7FC0 in K, 0xFFC0 in V): a read of a reserved slot poisons
    the output, and a missing append leaves a NaN behind;
  * ragged workloads draw pos_b uniformly from [lo, hi];
  * 8-bit caches (FP8 E4M3 or INT8 codes, one scale per KV head) are drawn as
    codes, not converted from values: E4M3 entries take every finite code
    (both signs, subnormals up to +-448) with equal probability, INT8 entries
    take [-127, 127] uniformly; the per-head scales are (0.5 + U[0, 1)) / 64
    for E4M3 and (0.5 + U[0, 1)) / 32 for INT8, as float32; reserved slots
    hold the E4M3 NaN codes (0x7F in K, 0xFF in V) or -128, which no INT8
    entry uses;
  * each tensor has its own stream: PCG64 seeded with
    SeedSequence([0xFA57, seed, workload index, layer, tensor id, chunk]).
    Large tensors are filled in fixed 4 Mi-element chunks, so the bits do not
    depend on the number of threads used to fill them.

This module draws random numbers and nothing else: it holds none of the
layer's arithmetic.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass
from typing import Dict

import numpy as np

from .configs import LayerConfig

SEED_DOMAIN = 0xFA57
K_SENTINEL = 0x7FC0
V_SENTINEL = 0xFFC0
CHUNK = 1 << 22

T_X, T_ATTN_NORM, T_WQ, T_WK, T_WV, T_WO, T_MLP_NORM, T_WG, T_WU, T_WD, T_KC, T_VC, T_POS = range(13)
T_KC8, T_VC8, T_KS, T_VS = range(13, 17)

KV8_FORMATS = ("fp8_e4m3", "int8")
K8_SENTINEL = {"fp8_e4m3": 0x7F, "int8": 0x80}
V8_SENTINEL = {"fp8_e4m3": 0xFF, "int8": 0x80}

WEIGHT_NAMES = ("attn_norm", "w_q", "w_k", "w_v", "w_o", "mlp_norm", "w_gate", "w_up", "w_down")


def fp32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 bit patterns (nearest, ties to even).

    Inputs here are finite draws, so no NaN/Inf handling is needed.
    """
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = u >> np.uint32(16)
    r &= np.uint32(1)
    r += np.uint32(0x7FFF)
    r += u
    r >>= np.uint32(16)
    return r.astype(np.uint16)


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _normal_bf16(seed_words, n: int, scale: float, mean: float = 0.0) -> np.ndarray:
    """n draws of mean + scale * N(0,1) as bf16 bits, filled chunk by chunk."""
    out = np.empty(n, dtype=np.uint16)
    nchunks = (n + CHUNK - 1) // CHUNK

    def fill(c):
        lo, hi = c * CHUNK, min(n, (c + 1) * CHUNK)
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(seed_words) + [c])))
        v = rng.standard_normal(hi - lo, dtype=np.float32)
        if scale != 1.0:
            v *= np.float32(scale)
        if mean != 0.0:
            v += np.float32(mean)
        out[lo:hi] = fp32_to_bf16_bits(v)

    if nchunks <= 1:
        for c in range(nchunks):
            fill(c)
    else:
        with ThreadPoolExecutor(max_workers=min(_threads(), nchunks)) as ex:
            list(ex.map(fill, range(nchunks)))
    return out


def _words(cfg: LayerConfig, seed: int, layer: int, tensor: int):
    return [SEED_DOMAIN, int(seed), int(cfg.index), int(layer), int(tensor)]


def make_pos(cfg: LayerConfig, seed: int = 0) -> np.ndarray:
    """Per-sequence positions N_p (int32 [B])."""
    if cfg.ragged is None:
        return np.asarray(cfg.pos, dtype=np.int32)
    lo, hi = cfg.ragged
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(_words(cfg, seed, 0, T_POS))))
    return rng.integers(lo, hi + 1, size=cfg.batch).astype(np.int32)


def make_x(cfg: LayerConfig, seed: int = 0) -> np.ndarray:
    """Token activations x, bf16 bits [B, D]."""
    return _normal_bf16(_words(cfg, seed, 0, T_X), cfg.batch * cfg.hidden, 1.0).reshape(cfg.batch, cfg.hidden)


def make_weights(cfg: LayerConfig, layer: int = 0, seed: int = 0) -> Dict[str, np.ndarray]:
    """Raw weights of one layer, bf16 bits, nn.Linear layout [out, in]."""
    D, K, q, kv = cfg.hidden, cfg.intermediate, cfg.q_dim, cfg.kv_dim
    spec = {
        "attn_norm": (T_ATTN_NORM, (D,), 0.1, 1.0),
        "w_q": (T_WQ, (q, D), 0.02, 0.0),
        "w_k": (T_WK, (kv, D), 0.02, 0.0),
        "w_v": (T_WV, (kv, D), 0.02, 0.0),
        "w_o": (T_WO, (D, q), 0.02, 0.0),
        "mlp_norm": (T_MLP_NORM, (D,), 0.1, 1.0),
        "w_gate": (T_WG, (K, D), 0.02, 0.0),
        "w_up": (T_WU, (K, D), 0.02, 0.0),
        "w_down": (T_WD, (D, K), 0.02, 0.0),
    }
    out = {}
    for name, (tid, shape, scale, mean) in spec.items():
        n = int(np.prod(shape))
        out[name] = _normal_bf16(_words(cfg, seed, layer, tid), n, scale, mean).reshape(shape)
    return out


def make_cache(cfg: LayerConfig, pos: np.ndarray, which: str, layer: int = 0, seed: int = 0) -> np.ndarray:
    """Static KV cache [B, H_kv, N_max, d] as bf16 bits.

    Entries [0, pos_b) are N(0,1) draws; every other slot holds the sentinel.
    """
    tid, sentinel = (T_KC, K_SENTINEL) if which == "k" else (T_VC, V_SENTINEL)
    B, G, N, d = cfg.batch, cfg.n_kv_heads, cfg.max_seq, cfg.head_dim
    cache = np.full((B, G, N, d), sentinel, dtype=np.uint16)
    for b in range(B):
        p = int(pos[b])
        if p <= 0:
            continue
        vals = _normal_bf16(_words(cfg, seed, layer, tid) + [b], G * p * d, 1.0)
        cache[b, :, :p, :] = vals.reshape(G, p, d)
    return cache


def _codes8(seed_words, n: int, fmt: str) -> np.ndarray:
    """n random 8-bit cache codes of the format, filled chunk by chunk."""
    out = np.empty(n, dtype=np.uint8)
    for c in range((n + CHUNK - 1) // CHUNK):
        lo, hi = c * CHUNK, min(n, (c + 1) * CHUNK)
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(seed_words) + [c])))
        if fmt == "fp8_e4m3":
            r = rng.integers(0, 254, size=hi - lo)       # 254 finite codes: skip 0x7F and 0xFF
            out[lo:hi] = np.where(r < 0x7F, r, r + 1).astype(np.uint8)
        elif fmt == "int8":
            out[lo:hi] = rng.integers(-127, 128, size=hi - lo).astype(np.int8).view(np.uint8)
        else:
            raise ValueError(f"unknown 8-bit format {fmt!r}")
    return out


def make_cache8(cfg: LayerConfig, pos: np.ndarray, which: str, fmt: str, layer: int = 0,
                seed: int = 0) -> np.ndarray:
    """8-bit KV cache [B, H_kv, N_max, d] of codes: random codes in [0, pos_b), the sentinel elsewhere."""
    tid, sentinel = (T_KC8, K8_SENTINEL[fmt]) if which == "k" else (T_VC8, V8_SENTINEL[fmt])
    B, G, N, d = cfg.batch, cfg.n_kv_heads, cfg.max_seq, cfg.head_dim
    cache = np.full((B, G, N, d), sentinel, dtype=np.uint8)
    for b in range(B):
        p = int(pos[b])
        if p <= 0:
            continue
        cache[b, :, :p, :] = _codes8(_words(cfg, seed, layer, tid) + [b], G * p * d, fmt).reshape(G, p, d)
    return cache


def make_kv_scales(cfg: LayerConfig, which: str, fmt: str, layer: int = 0, seed: int = 0) -> np.ndarray:
    """Per-KV-head scales of an 8-bit cache, float32 [H_kv]."""
    if fmt not in KV8_FORMATS:
        raise ValueError(f"unknown 8-bit format {fmt!r}")
    tid = T_KS if which == "k" else T_VS
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(_words(cfg, seed, layer, tid))))
    div = np.float32(64.0 if fmt == "fp8_e4m3" else 32.0)
    return ((np.float32(0.5) + rng.random(cfg.n_kv_heads, dtype=np.float32)) / div).astype(np.float32)


@dataclass
class LayerInputs:
    cfg: LayerConfig
    x: np.ndarray          # bf16 bits [B, D]
    pos: np.ndarray        # int32 [B]
    weights: Dict[str, np.ndarray]
    k_cache: np.ndarray    # bf16 bits [B, H_kv, N_max, d]
    v_cache: np.ndarray


def make_layer_inputs(cfg: LayerConfig, layer: int = 0, seed: int = 0, pos=None) -> LayerInputs:
    p = make_pos(cfg, seed) if pos is None else np.asarray(pos, dtype=np.int32)
    if p.shape != (cfg.batch,):
        raise ValueError(f"pos must have shape ({cfg.batch},), got {p.shape}")
    return LayerInputs(cfg=cfg, x=make_x(cfg, seed), pos=p,
                       weights=make_weights(cfg, layer, seed),
                       k_cache=make_cache(cfg, p, "k", layer, seed),
                       v_cache=make_cache(cfg, p, "v", layer, seed))
