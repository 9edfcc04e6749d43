"""Planted mistakes in the oracle must be caught by its pins (CPU only).

Each mutant is the oracle's source with one plausible slip (a flipped sign, a
dropped term, a wrong index, a transposed operand, a wrong rounding). The pins
of ``test_oracle_pins`` that do not depend on the oracle's own arithmetic
(brute force, hand-derived bf16 patterns, closed forms) are run against the
mutant, and at least one of them has to fail.
"""
import math
import os
import types

import numpy as np
import pytest

from oracle import brute
from paper_2607_11211_amd import inputs
from paper_2607_11211_amd.configs import LayerConfig

REF_PATH = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "ref.py")

MUTATIONS = {
    "rope_sign": ("a * c - b * s, b * c + a * s", "a * c + b * s, b * c - a * s"),
    "rope_freq": ("-2.0 * j / head_dim", "-1.0 * j / head_dim"),
    "rope_pos_off_by_one": ("k_r = rope(k, p, rope_base)", "k_r = rope(k, p + 1, rope_base)"),
    "rms_eps_outside": ("x / np.sqrt(ms + eps) * gamma", "x / (np.sqrt(ms) + eps) * gamma"),
    "rms_no_gamma": ("x / np.sqrt(ms + eps) * gamma", "x / np.sqrt(ms + eps)"),
    "rms_mean_abs": ("ms = np.mean(x * x, axis=-1, keepdims=True)",
                     "ms = np.mean(np.abs(x), axis=-1, keepdims=True) ** 2"),
    "attn_scale": ("s = (k @ q) / np.sqrt(float(d))", "s = (k @ q) / float(d)"),
    "gqa_strided": ("for hq in range(g * group, (g + 1) * group):", "for hq in range(g, H, G):"),
    "no_attn_residual": ('h1 = X[b] + linear(W["w_o"], o.reshape(H * d))',
                         'h1 = linear(W["w_o"], o.reshape(H * d))'),
    "mlp_residual_from_x": ("y = h1 + m", "y = X[b] + m"),
    "silu_sign": ("return z / (1.0 + np.exp(-z))", "return z / (1.0 + np.exp(z))"),
    "gate_up_swapped": ("a = silu(g) * u", "a = silu(u) * g"),
    "wq_transposed": ('q = linear(W["w_q"], h).reshape(H, d)', 'q = linear(W["w_q"].T, h).reshape(H, d)'),
    "unrounded_new_key": ("k_val(k_new[g], g)[None, :]", "k_r[g][None, :]"),
    "wrong_mlp_gain": ('h2 = rms_norm(h1, W["mlp_norm"], rms_eps)', 'h2 = rms_norm(h1, W["attn_norm"], rms_eps)'),
    "bf16_truncates": ("q = np.rint(np.ldexp(ax, -qexp))", "q = np.floor(np.ldexp(ax, -qexp))"),
    "bf16_ties_up": ("q = np.rint(np.ldexp(ax, -qexp))", "q = np.floor(np.ldexp(ax, -qexp) + 0.5)"),
}

CASES = [
    # square W_q (D = H d) so a transposed operand still type-checks
    LayerConfig(name="m1", index=200, batch=1, hidden=8, n_heads=2, n_kv_heads=1, head_dim=4,
                intermediate=6, rope_base=10000.0, max_seq=8, pos=(5,)),
    LayerConfig(name="m2", index=201, batch=2, hidden=8, n_heads=4, n_kv_heads=2, head_dim=2,
                intermediate=5, rope_base=10000.0, max_seq=8, pos=(3, 6)),
]


def load_mutant(old, new):
    src = open(REF_PATH).read()
    assert src.count(old) == 1, f"mutation anchor not unique: {old!r}"
    mod = types.ModuleType("oracle_ref_mutant")
    exec(compile(src.replace(old, new), "oracle_ref_mutant", "exec"), mod.__dict__)
    return mod


def pins(mod):
    """Pins that stand outside the oracle: brute force, golden bf16, closed forms."""
    for cfg in CASES:
        inp = inputs.make_layer_inputs(cfg)
        r = mod.decode_layer_cfg(cfg, inp.x, inp.pos, inp.k_cache, inp.v_cache, inp.weights)
        b = brute.decode_layer(inp.x.tolist(), inp.pos.tolist(), inp.k_cache.tolist(),
                               inp.v_cache.tolist(), {k: v.tolist() for k, v in inp.weights.items()},
                               n_heads=cfg.n_heads, n_kv_heads=cfg.n_kv_heads,
                               rope_base=cfg.rope_base, rms_eps=cfg.rms_eps)
        np.testing.assert_allclose(r["y"], np.array(b["y"]), rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(r["o"], np.array(b["o"]), rtol=1e-12, atol=1e-13)
        assert np.array_equal(r["k_new_bits"], np.array(b["k_new_bits"], dtype=np.uint16))
        assert np.array_equal(r["y_bits"], np.array(b["y_bits"], dtype=np.uint16))
    gold = os.path.join(os.path.dirname(__file__), "golden", "bf16_rne_cases.txt")
    for line in open(gold):
        line = line.strip()
        if line and not line.startswith("#"):
            v, bits = line.split()[:2]
            assert int(mod.f64_to_bf16_bits(np.array([float.fromhex(v)]))[0]) == int(bits, 16)
    out = mod.rope(np.array([1.0, 0.0]), 3, 10000.0)
    assert out[0] == pytest.approx(math.cos(3)) and out[1] == pytest.approx(math.sin(3))


def test_unmutated_oracle_passes_the_pins():
    pins(load_mutant("BF16_MAX =", "BF16_MAX ="))


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutant_is_caught(name):
    old, new = MUTATIONS[name]
    mod = load_mutant(old, new)
    with pytest.raises(Exception):
        pins(mod)
