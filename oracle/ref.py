"""fp64 reference of one token-phase decoder layer (FastTPS, Sections 2-3).

Test infrastructure only (see the package header). Every step is the plain
definition, evaluated in float64 on the exact values of the bf16 inputs; the
only roundings to bf16 are the ones the layer's storage boundary makes: the
K/V entries appended to the cache and the output token.

Readings of points the paper leaves open (each one is listed with its reason
in the design notes of the repository):
  * pre-norm residual block: h1 = x + W_o Attn(RMSNorm1(x)),
    y = h1 + MLP(RMSNorm2(h1)); no biases;
  * RMSNorm(x) = x / sqrt(mean(x^2) + eps) * gamma, eps inside the root;
  * RoPE is rotate-half: pairs (j, j + d/2), angle pos * base^(-2j/d), the
    same for every head, position = N_p (0-based index of the new token);
  * softmax scale 1/sqrt(d); the query attends exactly entries [0, N_p];
  * grouped-query attention: query head h reads KV head h // (H / H_kv);
  * attention consumes the appended K/V as stored, i.e. after bf16 rounding
    (after 8-bit quantization for an 8-bit cache, whose format is read in
    ``kvquant``).

Parity: pinned. Each function is checked by the CPU tests against brute force
in pure Python scalars, closed forms and invariants (RoPE group and
relative-position laws, softmax normalisation, one-entry attention, RMSNorm
scale law, SiLU identities, exact bf16 rounding against an exhaustive table),
and against the unfused formulations of Alg. 1 and Alg. 2.
"""
from __future__ import annotations

from typing import Dict, Mapping

import numpy as np

BF16_MAX = float.fromhex("0x1.fep127")  # largest finite bfloat16, bit pattern 0x7F7F


# ---------------------------------------------------------------------------
# bfloat16 storage boundary
# ---------------------------------------------------------------------------

def _widen_chunk(b: np.ndarray, out: np.ndarray) -> None:
    with np.errstate(invalid="ignore"):
        out[...] = (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_bits_to_f64(bits) -> np.ndarray:
    """Exact value of bf16 bit patterns (bfloat16 is the top half of binary32).

    Large arrays are widened in slices on a few threads; the result does not
    depend on the slicing (each element is converted on its own).
    """
    b = np.ascontiguousarray(np.asarray(bits, dtype=np.uint16))
    out = np.empty(b.shape, dtype=np.float64)
    n = b.size
    if n < (1 << 22):
        _widen_chunk(b, out)
        return out
    from concurrent.futures import ThreadPoolExecutor
    fb, fo = b.reshape(-1), out.reshape(-1)
    step = 1 << 21
    with ThreadPoolExecutor(max_workers=8) as ex:
        list(ex.map(lambda i: _widen_chunk(fb[i:i + step], fo[i:i + step]), range(0, n, step)))
    return out


def f64_to_bf16_bits(x) -> np.ndarray:
    """Round float64 values straight to bf16 (nearest, ties to even).

    The rounding is done once, from the float64 value: the significand is kept
    to 8 bits (binade quantum 2^(e-7)), with a fixed quantum of 2^-133 below
    the smallest normal 2^-126; results beyond the largest finite value become
    infinity; NaN becomes the quiet NaN 0x7FC0.
    """
    x = np.asarray(x, dtype=np.float64)
    ax = np.abs(x)
    with np.errstate(invalid="ignore", over="ignore"):
        _, e = np.frexp(ax)              # ax in [2^(e-1), 2^e)
        lead = e.astype(np.int64) - 1    # exponent of the leading bit
        qexp = np.maximum(lead, -126) - 7
        q = np.rint(np.ldexp(ax, -qexp))  # numpy rint rounds half to even
        r = np.ldexp(q, qexp)
        r = np.where(r > BF16_MAX, np.inf, r)
        r = np.where(np.isinf(ax), np.inf, r)
        signed = np.copysign(r, x)
        f32 = np.where(np.isnan(x), 0.0, signed).astype(np.float32)
    bits = (f32.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    return np.where(np.isnan(x), np.uint16(0x7FC0), bits).astype(np.uint16)


# ---------------------------------------------------------------------------
# operators (Section 2.2-2.3)
# ---------------------------------------------------------------------------

def rms_norm(x: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm over the last axis: x / sqrt(mean(x^2) + eps) * gamma.

    First step of the MLP block (Section 2.3 and Alg. 4); the same operator
    normalises the token before the QKV projection.
    """
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gamma


def linear(w: np.ndarray, v: np.ndarray) -> np.ndarray:
    """y = W v with W stored [out, in] (the projections of Section 2.2, Eq. mlp_main)."""
    return w @ v


def rope_inv_freq(head_dim: int, base: float) -> np.ndarray:
    """Frequencies base^(-2j/d), j = 0 .. d/2-1 (one per rotated pair)."""
    j = np.arange(head_dim // 2, dtype=np.float64)
    return np.power(float(base), -2.0 * j / head_dim)


def rope_cos_sin(pos: int, head_dim: int, base: float):
    """The sin/cos inputs of RoPE (Alg. 1 and Alg. 3 take them as d/2-long rows)."""
    theta = float(pos) * rope_inv_freq(head_dim, base)
    return np.cos(theta), np.sin(theta)


def rope(v: np.ndarray, pos: int, base: float) -> np.ndarray:
    """Rotary embedding of head vectors v[..., d] at position pos (rotate-half).

    Pair (j, j + d/2) is rotated by theta_j: (a, b) -> (a cos - b sin, b cos + a sin).
    Alg. 3 applies one RoPE call to Q and K together with shared sin/cos (Eq. 22);
    applying this function to both is the same computation.
    """
    d = v.shape[-1]
    half = d // 2
    c, s = rope_cos_sin(pos, d, base)
    a, b = v[..., :half], v[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def softmax(s: np.ndarray) -> np.ndarray:
    """Softmax over the last axis (the normalisation step of Alg. 1 and Eq. 26)."""
    z = np.exp(s - np.max(s, axis=-1, keepdims=True))
    return z / np.sum(z, axis=-1, keepdims=True)


def attention_one_query(q: np.ndarray, k: np.ndarray, v: np.ndarray):
    """One query row over n cached entries: S = q K^T / sqrt(d), P = softmax(S), O = P V.

    q [d], k and v [n, d]; Eq. 25, 26 and 28 with B = N = H = 1.
    Returns (o [d], p [n]).
    """
    d = q.shape[-1]
    s = (k @ q) / np.sqrt(float(d))
    p = softmax(s)
    return p @ v, p


def silu(z: np.ndarray) -> np.ndarray:
    """SiLU(z) = z / (1 + exp(-z))."""
    return z / (1.0 + np.exp(-z))


def mlp(h: np.ndarray, w_gate, w_up, w_down):
    """Eq. mlp_main: O = W_down (SiLU(W_gate h) * (W_up h)). Returns (O, gate, up, a)."""
    g = linear(w_gate, h)
    u = linear(w_up, h)
    a = silu(g) * u
    return linear(w_down, a), g, u, a


# ---------------------------------------------------------------------------
# GKVC: static cache with in-place append (Section 3.1.1, Eq. 1)
# ---------------------------------------------------------------------------

def gkvc_offset(b: int, g: int, n_p: int, n_kv_heads: int, max_seq: int, head_dim: int) -> int:
    """Element offset of the append slot (Eq. 1): h (N_p + N_r) d + N_p d with h = b H_kv + g.

    N_p + N_r is the fixed capacity max_seq of each (sequence, head) row.
    """
    h = b * n_kv_heads + g
    return h * max_seq * head_dim + n_p * head_dim


def gkvc_append(cache_bits: np.ndarray, pos, new_bits: np.ndarray) -> np.ndarray:
    """Copy of a [B, H_kv, N_max, d] cache with new[b, g] written at slot pos_b (Eq. 1).

    Every other element is left as it was; the counters move as the paper's
    update rule says (N_p <- N_p + 1, N_r <- N_r - 1), which the caller tracks.
    """
    out = np.array(cache_bits, copy=True)
    B, G, N, d = out.shape
    flat = out.reshape(-1)
    for b in range(B):
        p = int(pos[b])
        if not 0 <= p < N:
            raise ValueError(f"cache full or bad position: pos={p}, capacity={N}")
        for g in range(G):
            off = gkvc_offset(b, g, p, G, N, d)
            flat[off:off + d] = new_bits[b, g]
    return out


# ---------------------------------------------------------------------------
# one decode step of one layer
# ---------------------------------------------------------------------------

WEIGHT_KEYS = ("attn_norm", "w_q", "w_k", "w_v", "w_o", "mlp_norm", "w_gate", "w_up", "w_down")


def widen_weights(weights_bits: Mapping[str, np.ndarray]) -> Dict[str, np.ndarray]:
    """Exact float64 values of a layer's bf16 weights."""
    return {k: bf16_bits_to_f64(weights_bits[k]) for k in WEIGHT_KEYS}


def decode_layer(x_bits, pos, k_cache_bits, v_cache_bits, weights, *, n_heads: int,
                 n_kv_heads: int, rope_base: float, rms_eps: float, kv=None,
                 new_entries=None) -> Dict[str, np.ndarray]:
    """One token-phase step of one decoder layer, per sequence b.

    Inputs: x_bits [B, D] bf16 bits; pos [B] (N_p per sequence); caches
    [B, H_kv, N_max, d] bf16 bits holding entries [0, N_p); weights as bf16 bits
    in nn.Linear layout, or already widened by ``widen_weights``.

    With ``kv`` (a ``kvquant.KvQuant``: 8-bit format and per-KV-head scales)
    the caches hold 8-bit codes instead: a cached entry of KV head g is read as
    scale_g * value(code), and the entries appended in step 4 are the codes of
    k_rope / k_scale_g and v / v_scale_g. ``new_entries`` = (k, v), arrays
    [B, H_kv, d] of bits or codes, replaces the entries step 4 would append
    (teacher forcing: where a rounding of the GPU's own entry lands on the
    neighbouring value, the rest of the step is compared on that entry).

    Steps (Section 2.2 / Alg. 3 for attention, Eq. mlp_main for the MLP):
      1. h  = RMSNorm1(x)
      2. q, k, v = W_q h, W_k h, W_v h
      3. RoPE on q and k at position N_p
      4. k^, v^ = bf16(k_rope), bf16(v): the entries appended at slot N_p (Eq. 1)
      5. per query head: attention over the N_p cached entries and the new one
      6. h1 = x + W_o o
      7. h2 = RMSNorm2(h1)
      8. a  = SiLU(W_gate h2) * (W_up h2)
      9. y  = h1 + W_down a, and bf16(y)
    Returns every intermediate, float64 unless named *_bits.
    """
    if kv is not None:
        from . import kvquant
    W = weights if weights["w_q"].dtype == np.float64 else widen_weights(weights)
    X = bf16_bits_to_f64(x_bits)
    B, D = X.shape
    G = n_kv_heads
    H = n_heads
    d = k_cache_bits.shape[-1]
    group = H // G
    K = W["w_gate"].shape[0]
    out = {
        "h": np.zeros((B, D)), "q": np.zeros((B, H, d)), "k": np.zeros((B, G, d)),
        "v": np.zeros((B, G, d)), "q_rope": np.zeros((B, H, d)), "k_rope": np.zeros((B, G, d)),
        "k_new_bits": np.zeros((B, G, d), np.uint16 if kv is None else np.uint8),
        "v_new_bits": np.zeros((B, G, d), np.uint16 if kv is None else np.uint8),
        "o": np.zeros((B, H, d)), "h1": np.zeros((B, D)), "h2": np.zeros((B, D)),
        "gate": np.zeros((B, K)), "up": np.zeros((B, K)), "a": np.zeros((B, K)),
        "y": np.zeros((B, D)),
    }
    for b in range(B):
        p = int(pos[b])
        if not 0 <= p < k_cache_bits.shape[2]:
            raise ValueError(f"cache full or bad position: pos={p}")
        h = rms_norm(X[b], W["attn_norm"], rms_eps)
        q = linear(W["w_q"], h).reshape(H, d)
        k = linear(W["w_k"], h).reshape(G, d)
        v = linear(W["w_v"], h).reshape(G, d)
        q_r = rope(q, p, rope_base)
        k_r = rope(k, p, rope_base)
        if kv is None:
            k_new = f64_to_bf16_bits(k_r)
            v_new = f64_to_bf16_bits(v)
            k_val = v_val = lambda bits, g: bf16_bits_to_f64(bits)
        else:
            k_new = np.stack([kvquant.quantize(k_r[g], kv.k_scale[g], kv.fmt) for g in range(G)])
            v_new = np.stack([kvquant.quantize(v[g], kv.v_scale[g], kv.fmt) for g in range(G)])
            k_val = lambda codes, g: kvquant.dequantize(codes, kv.k_scale[g], kv.fmt)
            v_val = lambda codes, g: kvquant.dequantize(codes, kv.v_scale[g], kv.fmt)
        if new_entries is not None:
            k_new = np.asarray(new_entries[0][b], dtype=k_new.dtype)
            v_new = np.asarray(new_entries[1][b], dtype=v_new.dtype)
        o = np.zeros((H, d))
        for g in range(G):
            kc = np.concatenate([k_val(k_cache_bits[b, g, :p], g), k_val(k_new[g], g)[None, :]], axis=0)
            vc = np.concatenate([v_val(v_cache_bits[b, g, :p], g), v_val(v_new[g], g)[None, :]], axis=0)
            for hq in range(g * group, (g + 1) * group):
                o[hq], _ = attention_one_query(q_r[hq], kc, vc)
        h1 = X[b] + linear(W["w_o"], o.reshape(H * d))
        h2 = rms_norm(h1, W["mlp_norm"], rms_eps)
        m, gt, up, a = mlp(h2, W["w_gate"], W["w_up"], W["w_down"])
        y = h1 + m
        for name, val in (("h", h), ("q", q), ("k", k), ("v", v), ("q_rope", q_r),
                          ("k_rope", k_r), ("k_new_bits", k_new), ("v_new_bits", v_new),
                          ("o", o), ("h1", h1), ("h2", h2), ("gate", gt), ("up", up),
                          ("a", a), ("y", y)):
            out[name][b] = val
    out["y_bits"] = f64_to_bf16_bits(out["y"])
    return out


def decode_layer_cfg(cfg, x_bits, pos, k_cache_bits, v_cache_bits, weights, kv=None, new_entries=None):
    """decode_layer with the head counts, RoPE base and eps taken from a shape record."""
    return decode_layer(x_bits, pos, k_cache_bits, v_cache_bits, weights,
                        n_heads=cfg.n_heads, n_kv_heads=cfg.n_kv_heads,
                        rope_base=cfg.rope_base, rms_eps=cfg.rms_eps, kv=kv, new_entries=new_entries)
