"""Pins of the oracle's 8-bit KV cache formats and of the layer with an 8-bit cache (CPU only).

The E4M3 table is checked against its field definition written out by hand
(closed forms) and against torch.float8_e4m3fn, an implementation of the OCP
format independent of the oracle; the encoder against torch on float32
inputs, on every midpoint of the grid and on saturation; INT8 against
Python's round (ties to even) and the symmetric range. The layer with an
8-bit cache is pinned to the bf16 layer where both hold the same values, to
the nearest-code property of its appended entries, and to one-entry
attention. Planted mistakes in either module must be caught.
"""
import math
import os
import sys
import types

import numpy as np
import pytest
import torch

from oracle import kvquant as kq
from oracle import ref
from paper_2607_11211_amd import inputs
from paper_2607_11211_amd.configs import LayerConfig

ORACLE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle")


def torch_e4m3_values():
    return torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).double().numpy()


# ---------------------------------------------------------------------------
# E4M3 table
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("code,value", [
    (0x00, 0.0), (0x01, 2.0 ** -9), (0x07, 7 * 2.0 ** -9), (0x08, 2.0 ** -6), (0x30, 0.5),
    (0x38, 1.0), (0x3C, 1.5), (0x40, 2.0), (0x77, 240.0), (0x78, 256.0), (0x7E, 448.0),
    (0xB8, -1.0), (0xFE, -448.0), (0x81, -(2.0 ** -9)),
])
def test_e4m3_closed_forms(code, value):
    assert kq.E4M3_VALUES[code] == value


def test_e4m3_nan_and_negative_zero():
    assert math.isnan(kq.E4M3_VALUES[0x7F]) and math.isnan(kq.E4M3_VALUES[0xFF])
    assert kq.E4M3_VALUES[0x80] == 0.0 and math.copysign(1.0, kq.E4M3_VALUES[0x80]) == -1.0


def test_e4m3_table_equals_torch():
    t = torch_e4m3_values()
    nan = np.isnan(t)
    assert np.array_equal(np.isnan(kq.E4M3_VALUES), nan)
    assert np.array_equal(kq.E4M3_VALUES[~nan], t[~nan])


def test_e4m3_grid_monotone_symmetric():
    pos = kq.E4M3_VALUES[:0x7F]
    assert np.all(np.diff(pos) > 0)
    assert np.array_equal(kq.E4M3_VALUES[0x81:0xFF], -pos[1:])


# ---------------------------------------------------------------------------
# E4M3 rounding
# ---------------------------------------------------------------------------

def test_e4m3_round_equals_torch_on_float32():
    rng = np.random.default_rng(7)
    n = 100_000
    x = (rng.standard_normal(n) * np.exp(rng.uniform(-14, 7, n))).astype(np.float32)
    x = np.clip(x, np.float32(-448), np.float32(448))
    t = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(kq.e4m3_round(x.astype(np.float64)), t)


def test_e4m3_midpoints_tie_to_even_code():
    v = kq.E4M3_VALUES[:0x7F]
    mid = (v[:-1] + v[1:]) / 2.0            # exact in float64
    got = kq.e4m3_round(mid)
    lo = np.arange(0x7E, dtype=np.uint8)
    want = np.where(lo % 2 == 0, lo, lo + 1).astype(np.uint8)
    assert np.array_equal(got, want)
    assert np.array_equal(kq.e4m3_round(np.nextafter(mid, np.inf)), lo + 1)
    assert np.array_equal(kq.e4m3_round(np.nextafter(mid, -np.inf)), lo)
    assert np.array_equal(kq.e4m3_round(-mid), want | 0x80)


def test_e4m3_saturation_zero_and_sign():
    cases = [(448.0, 0x7E), (460.0, 0x7E), (464.0, 0x7E), (1e30, 0x7E), (np.inf, 0x7E), (-1e30, 0xFE),
             (0.0, 0x00), (-0.0, 0x80), (-1e-30, 0x80), (2.0 ** -10, 0x00), (3 * 2.0 ** -10, 0x02),
             (1.0625, 0x38), (1.1875, 0x3A), (432.0, 0x7E), (431.99, 0x7D)]
    for x, code in cases:
        assert int(kq.e4m3_round(np.array([x]))[0]) == code, x


def test_e4m3_round_is_nearest_exhaustive_search():
    rng = np.random.default_rng(8)
    x = rng.uniform(-500, 500, 4000) * np.exp(rng.uniform(-12, 0, 4000))
    c = kq.e4m3_round(x)
    got = kq.E4M3_VALUES[c]
    finite = kq.E4M3_VALUES[~np.isnan(kq.E4M3_VALUES)]
    best = np.min(np.abs(np.clip(x, -448, 448)[:, None] - finite[None, :]), axis=1)
    assert np.all(np.abs(np.clip(x, -448, 448) - got) == best)


# ---------------------------------------------------------------------------
# INT8
# ---------------------------------------------------------------------------

def test_int8_round_against_python_round():
    xs = np.arange(-1040, 1041) / 8.0     # quarter and eighth steps, many exact ties
    got = kq.int8_round(xs).view(np.int8).astype(int)
    want = np.array([max(-127, min(127, round(float(x)))) for x in xs])
    assert np.array_equal(got, want)


def test_int8_range_and_values():
    assert kq.int8_round(np.array([-1e9]))[0] == np.uint8(0x81)          # -127, never -128
    assert np.array_equal(kq.code_values(np.array([0x81, 0x7F, 0x00, 0xFF], np.uint8), kq.INT8),
                          [-127.0, 127.0, 0.0, -1.0])


# ---------------------------------------------------------------------------
# scaled codes
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("fmt", kq.FORMATS)
def test_quantize_error_within_half_step(fmt):
    rng = np.random.default_rng(9)
    s = 0.0371
    top = (448.0 if fmt == kq.FP8_E4M3 else 127.0) * s
    x = rng.uniform(-top, top, 20000)
    err = np.abs(kq.dequantize(kq.quantize(x, s, fmt), s, fmt) - x)
    assert np.all(err <= kq.grid_step(x, s, fmt) / 2 * (1 + 1e-12))


def test_grid_step_is_spacing_of_neighbours():
    v = kq.E4M3_VALUES[1:0x7F]
    # the spacing above each positive grid value (the last binade's spacing for 448)
    up = np.append(np.diff(v), 32.0)
    assert np.array_equal(kq.grid_step(v, 1.0, kq.FP8_E4M3), up)


# ---------------------------------------------------------------------------
# the layer with an 8-bit cache
# ---------------------------------------------------------------------------

def kv8_cfg(pos=(5,), n_heads=4, n_kv_heads=2, head_dim=4, index=300):
    return LayerConfig(name="kv8_tiny", index=index, batch=len(pos), hidden=8, n_heads=n_heads,
                       n_kv_heads=n_kv_heads, head_dim=head_dim, intermediate=6, rope_base=10000.0,
                       max_seq=8, pos=tuple(pos))


def pow2_kv(fmt, G):
    # distinct powers of two per head and between K and V: scaled codes stay exact in bf16
    return kq.KvQuant(fmt, tuple(2.0 ** -(4 + g) for g in range(G)), tuple(2.0 ** -(2 + 2 * g) for g in range(G)))


def caches8(cfg, inp, fmt):
    return (inputs.make_cache8(cfg, inp.pos, "k", fmt), inputs.make_cache8(cfg, inp.pos, "v", fmt))


def bf16_of_dequantized(codes, scales, fmt, pos, sentinel):
    out = np.full(codes.shape, sentinel, np.uint16)
    for b in range(codes.shape[0]):
        for g in range(codes.shape[1]):
            p = int(pos[b])
            vals = kq.dequantize(codes[b, g, :p], scales[g], fmt)
            bits = ref.f64_to_bf16_bits(vals)
            assert np.array_equal(ref.bf16_bits_to_f64(bits), vals)  # exact in bf16
            out[b, g, :p] = bits
    return out


def layer_pins(mod_ref, fmt):
    """The layer with an 8-bit cache against facts outside its kv path."""
    for cfg in (kv8_cfg(), kv8_cfg(pos=(3, 6), n_heads=2, n_kv_heads=2, head_dim=2, index=301)):
        inp = inputs.make_layer_inputs(cfg)
        kc8, vc8 = caches8(cfg, inp, fmt)
        G = cfg.n_kv_heads
        kv = pow2_kv(fmt, G)
        # (1) W_k = W_v = 0: the new entries are zero in both layers, so the
        # 8-bit layer equals the bf16 layer on the dequantized caches exactly
        w0 = dict(inp.weights)
        w0["w_k"] = np.zeros_like(w0["w_k"])
        w0["w_v"] = np.zeros_like(w0["w_v"])
        kb = bf16_of_dequantized(kc8, kv.k_scale, fmt, inp.pos, inputs.K_SENTINEL)
        vb = bf16_of_dequantized(vc8, kv.v_scale, fmt, inp.pos, inputs.V_SENTINEL)
        r8 = mod_ref.decode_layer_cfg(cfg, inp.x, inp.pos, kc8, vc8, w0, kv=kv)
        rb = ref.decode_layer_cfg(cfg, inp.x, inp.pos, kb, vb, w0)
        for key in ("o", "h1", "y"):
            assert np.array_equal(r8[key], rb[key]), key
        # (1b) the same with forced new entries: random codes in the 8-bit
        # layer, their exact values as bf16 in the bf16 layer
        rng = np.random.default_rng(cfg.index)
        fk = rng.integers(0, 256, (cfg.batch, G, cfg.head_dim)).astype(np.uint8)
        fv = rng.integers(0, 256, (cfg.batch, G, cfg.head_dim)).astype(np.uint8)
        if fmt == kq.FP8_E4M3:
            fk[(fk & 0x7F) == 0x7F] = 0x7E
            fv[(fv & 0x7F) == 0x7F] = 0xFE
        else:
            fk[fk == 0x80] = 0x81
            fv[fv == 0x80] = 0x81
        fkb = np.stack([[ref.f64_to_bf16_bits(kq.dequantize(fk[b, g], kv.k_scale[g], fmt)) for g in range(G)]
                        for b in range(cfg.batch)])
        fvb = np.stack([[ref.f64_to_bf16_bits(kq.dequantize(fv[b, g], kv.v_scale[g], fmt)) for g in range(G)]
                        for b in range(cfg.batch)])
        r8 = mod_ref.decode_layer_cfg(cfg, inp.x, inp.pos, kc8, vc8, inp.weights, kv=kv, new_entries=(fk, fv))
        rb = ref.decode_layer_cfg(cfg, inp.x, inp.pos, kb, vb, inp.weights, new_entries=(fkb, fvb))
        for key in ("o", "h1", "y"):
            assert np.array_equal(r8[key], rb[key]), key
        # (2) the appended codes are the nearest codes of k_rope / s and v / s,
        # with k_rope and v from the bf16 layer (same upstream arithmetic)
        r8 = mod_ref.decode_layer_cfg(cfg, inp.x, inp.pos, kc8, vc8, inp.weights, kv=kv)
        rb = ref.decode_layer_cfg(cfg, inp.x, inp.pos, inp.k_cache, inp.v_cache, inp.weights)
        allc = np.array([c for c in range(256) if not np.isnan(kq.code_values(np.uint8(c), fmt))], np.uint8)
        grid = kq.code_values(allc, fmt)
        for name, x, sc in (("k_new_bits", rb["k_rope"], kv.k_scale), ("v_new_bits", rb["v"], kv.v_scale)):
            for b in range(cfg.batch):
                for g in range(G):
                    y = x[b, g] / sc[g]
                    got = kq.code_values(r8[name][b, g], fmt)
                    lim = 448.0 if fmt == kq.FP8_E4M3 else 127.0
                    best = np.min(np.abs(np.clip(y, -lim, lim)[:, None] - grid[None, :]), axis=1)
                    assert np.all(np.abs(np.clip(y, -lim, lim) - got) == best), name
    # (3) pos 0: one-entry attention returns the dequantized new V of the head's group
    cfg = kv8_cfg(pos=(0,), index=302)
    inp = inputs.make_layer_inputs(cfg)
    kc8, vc8 = caches8(cfg, inp, fmt)
    kv = pow2_kv(fmt, cfg.n_kv_heads)
    r8 = mod_ref.decode_layer_cfg(cfg, inp.x, inp.pos, kc8, vc8, inp.weights, kv=kv)
    group = cfg.n_heads // cfg.n_kv_heads
    for h in range(cfg.n_heads):
        g = h // group
        want = kv.v_scale[g] * kq.code_values(r8["v_new_bits"][0, g], fmt)
        np.testing.assert_allclose(r8["o"][0, h], want, rtol=1e-15, atol=0)
    # (4) forced entries replace the appended ones
    forced_v = np.full_like(r8["v_new_bits"], 0x38 if fmt == kq.FP8_E4M3 else 0x01)
    rf = mod_ref.decode_layer_cfg(cfg, inp.x, inp.pos, kc8, vc8, inp.weights, kv=kv,
                                  new_entries=(r8["k_new_bits"], forced_v))
    for h in range(cfg.n_heads):
        np.testing.assert_allclose(rf["o"][0, h], kv.v_scale[h // group], rtol=1e-15)


@pytest.mark.parametrize("fmt", kq.FORMATS)
def test_layer_kv8_pins(fmt):
    layer_pins(ref, fmt)


def test_kvquant_rejects_bad_scales_and_formats():
    with pytest.raises(ValueError):
        kq.KvQuant("fp8_e5m2", (1.0,), (1.0,))
    with pytest.raises(ValueError):
        kq.KvQuant(kq.INT8, (0.0,), (1.0,))
    with pytest.raises(ValueError):
        kq.KvQuant(kq.INT8, (1.0,), (float("nan"),))


# ---------------------------------------------------------------------------
# planted mistakes
# ---------------------------------------------------------------------------

def load(path, old, new, name):
    src = open(path).read()
    assert src.count(old) == 1, f"mutation anchor not unique: {old!r}"
    mod = types.ModuleType(name)
    mod.__package__ = "oracle"
    sys.modules[name] = mod  # dataclasses look their module up there
    try:
        exec(compile(src.replace(old, new), name, "exec"), mod.__dict__)
    finally:
        del sys.modules[name]
    return mod


def kvquant_pins(mod):
    t = torch_e4m3_values()
    nan = np.isnan(t)
    assert np.array_equal(mod.E4M3_VALUES[~nan], t[~nan])
    rng = np.random.default_rng(11)
    x = np.clip((rng.standard_normal(20000) * np.exp(rng.uniform(-14, 7, 20000))).astype(np.float32), -448, 448)
    tt = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(mod.e4m3_round(x.astype(np.float64)), tt)
    assert list(mod.e4m3_round(np.array([1e6, np.inf, -np.inf]))) == [0x7E, 0x7E, 0xFE]
    v = mod.E4M3_VALUES[:0x7F]
    lo = np.arange(0x7E, dtype=np.uint8)
    assert np.array_equal(mod.e4m3_round((v[:-1] + v[1:]) / 2), np.where(lo % 2 == 0, lo, lo + 1))
    xs = np.arange(-1040, 1041) / 8.0
    assert np.array_equal(mod.int8_round(xs).view(np.int8).astype(int),
                          [max(-127, min(127, round(float(q)))) for q in xs])


KVQUANT_MUTATIONS = {
    "e4m3_bias_8": ("* 2.0 ** (e - 7)", "* 2.0 ** (e - 8)"),
    "e4m3_subnormal_scale": ("(m / 8.0) * 2.0 ** -6", "(m / 8.0) * 2.0 ** -7"),
    "e4m3_ties_to_lower": ("pick = np.where(even.any(axis=-1, keepdims=True), even, cand)", "pick = cand"),
    "e4m3_no_saturation": ("ax = np.minimum(np.abs(x), E4M3_MAX)", "ax = np.abs(x)"),
    "int8_ties_away": ("np.clip(np.rint(np.asarray(x, dtype=np.float64)), -INT8_MAX, INT8_MAX)",
                       "np.clip(np.trunc(np.asarray(x, dtype=np.float64) + np.copysign(0.5, x)), -INT8_MAX, INT8_MAX)"),
    "int8_range_128": ("-INT8_MAX, INT8_MAX).astype(np.int8)", "-INT8_MAX - 1, INT8_MAX).astype(np.int8)"),
}

REF_KV_MUTATIONS = {
    "kv_scales_swapped": ("kvquant.dequantize(codes, kv.v_scale[g], kv.fmt)",
                          "kvquant.dequantize(codes, kv.k_scale[g], kv.fmt)"),
    "kv_scale_head0": ("k_val = lambda codes, g: kvquant.dequantize(codes, kv.k_scale[g], kv.fmt)",
                       "k_val = lambda codes, g: kvquant.dequantize(codes, kv.k_scale[0], kv.fmt)"),
    "kv_quantize_before_rope": ("kvquant.quantize(k_r[g], kv.k_scale[g], kv.fmt)",
                                "kvquant.quantize(k[g], kv.k_scale[g], kv.fmt)"),
    "kv_new_entry_unscaled": ("k_val(k_new[g], g)[None, :]", "kvquant.code_values(k_new[g], kv.fmt)[None, :]"),
    "kv_forced_ignored": ("k_new = np.asarray(new_entries[0][b], dtype=k_new.dtype)\n            v_new = np.asarray(new_entries[1][b], dtype=v_new.dtype)",
                          "pass"),
}


def test_unmutated_modules_pass():
    kvquant_pins(load(os.path.join(ORACLE, "kvquant.py"), "E4M3_MAX = 448.0", "E4M3_MAX = 448.0", "kvq_same"))
    mod = load(os.path.join(ORACLE, "ref.py"), "BF16_MAX =", "BF16_MAX =", "ref_same")
    for fmt in kq.FORMATS:
        layer_pins(mod, fmt)


@pytest.mark.parametrize("name", sorted(KVQUANT_MUTATIONS))
def test_kvquant_mutant_is_caught(name):
    old, new = KVQUANT_MUTATIONS[name]
    mod = load(os.path.join(ORACLE, "kvquant.py"), old, new, "kvq_mutant")
    with pytest.raises(Exception):
        kvquant_pins(mod)


@pytest.mark.parametrize("name", sorted(REF_KV_MUTATIONS))
def test_ref_kv_mutant_is_caught(name):
    old, new = REF_KV_MUTATIONS[name]
    mod = load(os.path.join(ORACLE, "ref.py"), old, new, "ref_kv_mutant")
    with pytest.raises(Exception):
        for fmt in kq.FORMATS:
            layer_pins(mod, fmt)
