"""8-bit KV cache formats for the fp64 oracle (test infrastructure only).

The paper states that its cache management works unchanged with a quantized
KV cache (Section 5.2, Compatibility with Acceleration Algorithm; Section 2.4,
Operator Type and OI, counts the concatenation of a quantized cache among the
memory-reorganisation operators) but fixes no format. The reading used here:

  * an entry's d values are stored as 8-bit codes, FP8 E4M3 (the OCP
    "e4m3fn" encoding: 1 sign, 4 exponent bits with bias 7, 3 mantissa bits;
    subnormals; no infinities; S.1111.111 is NaN; largest finite 448) or INT8
    (two's complement, symmetric range [-127, 127]);
  * one fp32 scale per (layer, KV head) for K and one for V, chosen by the
    caller; an entry's value is scale * value(code);
  * the entry appended at slot N_p (Eq. 1) is the code of k_rope / scale
    (v / scale), rounded to the nearest code, ties to the even code, values
    beyond the largest finite magnitude saturating to it. Rounding, division
    and the choice of code are all made once, from the float64 value.

Parity: pinned. The E4M3 table is checked against closed forms of the field
definition and against torch.float8_e4m3fn, the encoder against
torch.float8_e4m3fn on float32 inputs and against every midpoint of the grid,
the INT8 encoder against numpy rint and its range, and the layer with an
8-bit cache against the bf16 layer on equal cache values (tests of the CPU
suite).
"""
from __future__ import annotations

import dataclasses

import numpy as np

FP8_E4M3 = "fp8_e4m3"
INT8 = "int8"
FORMATS = (FP8_E4M3, INT8)
E4M3_MAX = 448.0
INT8_MAX = 127


def e4m3_value(code: int) -> float:
    """Value of an E4M3 code from its fields: (-1)^s 2^(e-7) (1 + m/8), or 2^-6 (m/8) when e = 0."""
    code = int(code) & 0xFF
    s, e, m = code >> 7, (code >> 3) & 0xF, code & 0x7
    if e == 0xF and m == 0x7:
        return float("nan")
    mag = (m / 8.0) * 2.0 ** -6 if e == 0 else (1.0 + m / 8.0) * 2.0 ** (e - 7)
    return -mag if s else mag


E4M3_VALUES = np.array([e4m3_value(c) for c in range(256)], dtype=np.float64)
# the non-negative finite codes 0x00..0x7E in increasing order of value
_POS_CODES = np.arange(0x7F, dtype=np.uint8)
_POS_VALUES = E4M3_VALUES[:0x7F]


def e4m3_round(x) -> np.ndarray:
    """Codes of float64 values: the nearest finite E4M3 value, ties to the code with an even last bit.

    |x| at or beyond the largest finite value gives +-448 (saturation); the
    sign bit is the sign of x, so a negative value that rounds to zero gives
    the code of -0 (0x80). NaN inputs are outside the contract.
    """
    x = np.asarray(x, dtype=np.float64)
    ax = np.minimum(np.abs(x), E4M3_MAX)
    # distance to every non-negative grid value; the nearest wins, ties go to the even code
    dist = np.abs(ax[..., None] - _POS_VALUES)
    best = dist.min(axis=-1, keepdims=True)
    cand = dist == best
    even = cand & ((_POS_CODES & 1) == 0)
    pick = np.where(even.any(axis=-1, keepdims=True), even, cand)
    code = np.argmax(pick, axis=-1).astype(np.uint8)
    return np.where(np.signbit(x), code | np.uint8(0x80), code).astype(np.uint8)


def int8_round(x) -> np.ndarray:
    """INT8 codes (as uint8 bit patterns) of float64 values: rint (ties to even), clamped to [-127, 127]."""
    q = np.clip(np.rint(np.asarray(x, dtype=np.float64)), -INT8_MAX, INT8_MAX).astype(np.int8)
    return q.view(np.uint8)


def code_values(codes, fmt: str) -> np.ndarray:
    """float64 values of 8-bit codes (without the scale)."""
    c = np.asarray(codes, dtype=np.uint8)
    if fmt == FP8_E4M3:
        return E4M3_VALUES[c]
    if fmt == INT8:
        return c.view(np.int8).astype(np.float64)
    raise ValueError(f"unknown KV format {fmt!r}")


def quantize(x, scale: float, fmt: str) -> np.ndarray:
    """Codes of x / scale (one KV head's scale)."""
    y = np.asarray(x, dtype=np.float64) / float(scale)
    if fmt == FP8_E4M3:
        return e4m3_round(y)
    if fmt == INT8:
        return int8_round(y)
    raise ValueError(f"unknown KV format {fmt!r}")


def dequantize(codes, scale: float, fmt: str) -> np.ndarray:
    """Values scale * value(code) of one KV head's codes."""
    return float(scale) * code_values(codes, fmt)


def grid_step(x, scale: float, fmt: str) -> np.ndarray:
    """Spacing of the scaled grid at |x|: the largest distance of x from a correctly chosen neighbour code.

    E4M3: 2^(e-3) in the binade [2^e, 2^(e+1)) for e >= -6, 2^-9 below;
    INT8: 1. Times the scale.
    """
    a = np.abs(np.asarray(x, dtype=np.float64)) / float(scale)
    if fmt == INT8:
        return np.full(a.shape, float(scale))
    with np.errstate(divide="ignore"):
        e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    e = np.clip(e, -6, 8)
    return float(scale) * np.ldexp(1.0, (e - 3).astype(np.int64))


@dataclasses.dataclass(frozen=True)
class KvQuant:
    """An 8-bit cache's format and per-KV-head scales (float32 values, held as float64)."""
    fmt: str
    k_scale: tuple
    v_scale: tuple

    def __post_init__(self):
        if self.fmt not in FORMATS:
            raise ValueError(f"unknown KV format {self.fmt!r}")
        for s in tuple(self.k_scale) + tuple(self.v_scale):
            if not (np.isfinite(s) and s > 0):
                raise ValueError("scales must be positive and finite")
