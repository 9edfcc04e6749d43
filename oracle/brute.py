"""The decode-step layer again, in pure Python scalars, for tiny shapes.

Test infrastructure only (see the package header). Written independently of
``ref``: no numpy, every sum is ``math.fsum``, bf16 bit patterns are decoded
from their sign/exponent/fraction fields, and rounding to bf16 is done exactly
with ``fractions.Fraction`` (nearest, ties to even). It follows the same
definitions and readings as ``ref`` (Sections 2.2-3.2, Eq. 1, Eq. mlp_main);
agreement to ~1e-12 relative pins the vectorised oracle.

Parity: this module is itself a pin; it is checked against hand-derived bit
patterns and against the invariants in the CPU tests.
"""
from __future__ import annotations

import math
from fractions import Fraction


def bf16_value(bits: int) -> float:
    """Value of a bf16 pattern from its fields: 1 sign, 8 exponent, 7 fraction bits."""
    bits = int(bits) & 0xFFFF
    sign = -1.0 if bits >> 15 else 1.0
    e = (bits >> 7) & 0xFF
    f = bits & 0x7F
    if e == 0xFF:
        return sign * math.inf if f == 0 else math.nan
    if e == 0:
        return sign * math.ldexp(f, -133)       # 2^-126 * f/128
    return sign * math.ldexp(128 + f, e - 127 - 7)


def bf16_round(x: float) -> int:
    """bf16 pattern nearest to x (ties to even), computed exactly."""
    if math.isnan(x):
        return 0x7FC0
    sign = 1 if math.copysign(1.0, x) < 0 else 0
    ax = abs(x)
    if math.isinf(ax):
        return (sign << 15) | 0x7F80
    if ax == 0.0:
        return sign << 15
    m, e = math.frexp(ax)                 # ax = m 2^e, 0.5 <= m < 1
    lead = e - 1
    qexp = max(lead, -126) - 7
    q = Fraction(ax) / Fraction(2) ** qexp
    n = math.floor(q)
    rem = q - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    # n * 2^qexp is the rounded magnitude; encode it
    if n == 0:
        return sign << 15
    if qexp == -133 and n < 128:          # subnormal
        return (sign << 15) | n
    if n == 256:                          # carried into the next binade
        n = 128
        qexp += 1
    biased = qexp + 7 + 127
    if biased >= 0xFF:
        return (sign << 15) | 0x7F80
    return (sign << 15) | (biased << 7) | (n - 128)


def _dot(a, b):
    return math.fsum(x * y for x, y in zip(a, b))


def _matvec(w, v):
    return [_dot(row, v) for row in w]


def _rms_norm(x, gamma, eps):
    ms = math.fsum(t * t for t in x) / len(x)
    r = 1.0 / math.sqrt(ms + eps)
    return [t * r * g for t, g in zip(x, gamma)]


def _rope(v, pos, base):
    d = len(v)
    half = d // 2
    out = [0.0] * d
    for j in range(half):
        th = pos * base ** (-2.0 * j / d)
        c, s = math.cos(th), math.sin(th)
        a, b = v[j], v[j + half]
        out[j] = a * c - b * s
        out[j + half] = b * c + a * s
    return out


def _silu(z):
    return z / (1.0 + math.exp(-z))


def decode_layer(x_bits, pos, k_cache_bits, v_cache_bits, weights, *, n_heads, n_kv_heads,
                 rope_base, rms_eps):
    """Same contract as ``ref.decode_layer``; nested Python lists in, dict of lists out.

    x_bits [B][D]; caches [B][H_kv][N_max][d]; weights as nested lists of bf16
    patterns in [out][in] layout.
    """
    W = {k: ([bf16_value(t) for t in w] if not isinstance(w[0], (list, tuple))
             else [[bf16_value(t) for t in row] for row in w]) for k, w in weights.items()}
    H, G = n_heads, n_kv_heads
    group = H // G
    res = {k: [] for k in ("q_rope", "k_new_bits", "v_new_bits", "o", "h1", "a", "y", "y_bits")}
    for b, xb in enumerate(x_bits):
        x = [bf16_value(t) for t in xb]
        p = int(pos[b])
        h = _rms_norm(x, W["attn_norm"], rms_eps)
        q = _matvec(W["w_q"], h)
        k = _matvec(W["w_k"], h)
        v = _matvec(W["w_v"], h)
        d = len(q) // H
        qr = [_rope(q[i * d:(i + 1) * d], p, rope_base) for i in range(H)]
        kr = [_rope(k[i * d:(i + 1) * d], p, rope_base) for i in range(G)]
        kn = [[bf16_round(t) for t in kr[g]] for g in range(G)]
        vn = [[bf16_round(t) for t in v[g * d:(g + 1) * d]] for g in range(G)]
        o = []
        for hq in range(H):
            g = hq // group
            keys = [[bf16_value(t) for t in k_cache_bits[b][g][j]] for j in range(p)]
            keys.append([bf16_value(t) for t in kn[g]])
            vals = [[bf16_value(t) for t in v_cache_bits[b][g][j]] for j in range(p)]
            vals.append([bf16_value(t) for t in vn[g]])
            scale = 1.0 / math.sqrt(d)
            s = [_dot(qr[hq], kk) * scale for kk in keys]
            mx = max(s)
            e = [math.exp(t - mx) for t in s]
            z = math.fsum(e)
            pr = [t / z for t in e]
            o.append([math.fsum(pr[j] * vals[j][i] for j in range(len(vals))) for i in range(d)])
        of = [t for row in o for t in row]
        attn = _matvec(W["w_o"], of)
        h1 = [a + c for a, c in zip(x, attn)]
        h2 = _rms_norm(h1, W["mlp_norm"], rms_eps)
        gt = _matvec(W["w_gate"], h2)
        up = _matvec(W["w_up"], h2)
        a = [_silu(g_) * u_ for g_, u_ in zip(gt, up)]
        mo = _matvec(W["w_down"], a)
        y = [c + m for c, m in zip(h1, mo)]
        for key, val in (("q_rope", qr), ("k_new_bits", kn), ("v_new_bits", vn), ("o", o),
                         ("h1", h1), ("a", a), ("y", y), ("y_bits", [bf16_round(t) for t in y])):
            res[key].append(val)
    return res
