"""Workload shapes for one token-phase decoder layer.

The shapes follow the model table of the FastTPS paper (Section 4.1, Faster Attention Block, Table 1):
the Phi-3-mini column gives 32 query heads = 32 KV heads, head dim 96, MLP width
8192 (hidden 3072 = 32 x 96); the Llama3 column gives 32 query heads over 8 KV
heads, head dim 128, MLP width 14336. Every workload here is synthetic: weights,
activations and cache contents are seeded random numbers (see ``inputs.py``).

This module holds sizes only; it does no arithmetic of the method.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Dict, Optional, Tuple


@dataclass(frozen=True)
class LayerConfig:
    """Shape of one decode step of one decoder layer.

    ``pos`` is the per-sequence position N_p of the new token (the number of
    entries already held in the static KV cache, Section 3.1.1); the step
    attends over ``pos + 1`` entries. ``max_seq`` is the cache capacity
    N_p + N_r per sequence (Eq. 1).
    """

    name: str
    index: int            # seed domain of the workload
    batch: int            # B
    hidden: int           # D
    n_heads: int          # H (query heads)
    n_kv_heads: int       # H_kv
    head_dim: int         # d
    intermediate: int     # K (MLP width)
    rope_base: float
    max_seq: int          # N_max
    pos: Tuple[int, ...]  # N_p per sequence (len == batch)
    layers: int = 1
    rms_eps: float = 1e-5
    # ragged lengths: pos drawn uniformly from [lo, hi] per sequence (seeded)
    ragged: Optional[Tuple[int, int]] = None

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def qkv_rows(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def group(self) -> int:
        return self.n_heads // self.n_kv_heads

    def weight_elems(self) -> int:
        D, K = self.hidden, self.intermediate
        return (self.qkv_rows * D + D * self.q_dim + 2 * K * D + K * D + 2 * D)

    def weight_bytes(self) -> int:
        """bf16 bytes of one layer's weights, each counted once."""
        return 2 * self.weight_elems()

    def kv_read_bytes(self, pos=None) -> int:
        """bf16 bytes of K and V read over the pre-existing entries [0, pos_b)."""
        p = self.pos if pos is None else pos
        return 2 * 2 * self.head_dim * self.n_kv_heads * int(sum(p))

    def step_bytes(self, pos=None) -> int:
        """Algorithmic HBM bytes of one layer step: weights + KV read."""
        return self.weight_bytes() + self.kv_read_bytes(pos)

    def with_pos(self, pos) -> "LayerConfig":
        return replace(self, pos=tuple(int(p) for p in pos))


def _phi3(name, index, pos, max_seq, batch=1, layers=1, ragged=None):
    return LayerConfig(name=name, index=index, batch=batch, hidden=3072,
                       n_heads=32, n_kv_heads=32, head_dim=96,
                       intermediate=8192, rope_base=10000.0, max_seq=max_seq,
                       pos=tuple([pos] * batch), layers=layers, ragged=ragged)


CONFIGS: Dict[str, LayerConfig] = {
    # tiny layer: D=256, 4x64 MHA, K=688, 128 entries prefilled, new token at 128
    "tiny": LayerConfig(name="tiny", index=0, batch=1, hidden=256, n_heads=4,
                        n_kv_heads=4, head_dim=64, intermediate=688,
                        rope_base=10000.0, max_seq=256, pos=(128,)),
    # Phi-3-mini-shaped layer, KV length 1024
    "phi3_kv1k": _phi3("phi3_kv1k", 1, 1024, 1152),
    # Phi-3-mini-shaped 32-layer stack, KV length 4096 per layer
    "phi3_stack32_kv4k": _phi3("phi3_stack32_kv4k", 2, 4096, 4224, layers=32),
    # 16 sequences, ragged KV lengths U[512, 4096]
    "phi3_batch16_ragged": _phi3("phi3_batch16_ragged", 3, 0, 4224, batch=16,
                                 ragged=(512, 4096)),
    # long-context GQA layer: D=4096, 32 q heads / 8 KV heads x 128, K=14336
    "gqa_longctx": LayerConfig(name="gqa_longctx", index=4, batch=4, hidden=4096,
                               n_heads=32, n_kv_heads=8, head_dim=128,
                               intermediate=14336, rope_base=500000.0,
                               max_seq=32896, pos=(32768,) * 4),
    # one layer of the 32-layer stack (Phi-3-mini shape at KV length 4096)
    "phi3_kv4k": _phi3("phi3_kv4k", 2, 4096, 4224),
}


def get(name: str) -> LayerConfig:
    try:
        return CONFIGS[name]
    except KeyError:
        raise KeyError(f"unknown config {name!r}; known: {sorted(CONFIGS)}") from None
