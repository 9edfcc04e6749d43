"""Pins of the fp64 oracle against facts outside itself (CPU only).

Each test checks the oracle against something the paper or the mathematics
fixes: hand-derived bf16 patterns, an exhaustive bf16 table, brute force in
pure Python scalars, closed forms (RoPE group law, one-entry attention),
invariants (norm preservation, softmax normalisation, permutation and
relative-position invariance, RMSNorm scale law) and the paper's equivalence
of its fused and unfused formulations (Section 3: Alg. 1 vs Alg. 3, Alg. 2 vs
Alg. 4).
"""
import math
import os

import numpy as np
import pytest

from oracle import brute, formulations, ref
from paper_2607_11211_amd import inputs
from paper_2607_11211_amd.configs import LayerConfig

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def tiny_cfg(hidden=8, n_heads=2, n_kv_heads=1, head_dim=4, intermediate=6, max_seq=8,
             pos=(5,), base=10000.0, index=100, eps=1e-5):
    return LayerConfig(name="brute_tiny", index=index, batch=len(pos), hidden=hidden,
                       n_heads=n_heads, n_kv_heads=n_kv_heads, head_dim=head_dim,
                       intermediate=intermediate, rope_base=base, max_seq=max_seq,
                       pos=tuple(pos), rms_eps=eps)


def run_ref(cfg, inp):
    return ref.decode_layer_cfg(cfg, inp.x, inp.pos, inp.k_cache, inp.v_cache, inp.weights)


def run_brute(cfg, inp):
    return brute.decode_layer(inp.x.tolist(), inp.pos.tolist(), inp.k_cache.tolist(),
                              inp.v_cache.tolist(), {k: v.tolist() for k, v in inp.weights.items()},
                              n_heads=cfg.n_heads, n_kv_heads=cfg.n_kv_heads,
                              rope_base=cfg.rope_base, rms_eps=cfg.rms_eps)


# ---------------------------------------------------------------------------
# bf16 boundary
# ---------------------------------------------------------------------------

def load_bf16_cases():
    cases = []
    with open(os.path.join(GOLDEN, "bf16_rne_cases.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            parts = line.split()
            cases.append((float.fromhex(parts[0]), int(parts[1], 16)))
    return cases


@pytest.mark.parametrize("value,bits", load_bf16_cases())
def test_bf16_golden_rounding(value, bits):
    assert int(ref.f64_to_bf16_bits(np.array([value]))[0]) == bits
    assert brute.bf16_round(value) == bits


def test_bf16_decode_exhaustive():
    allb = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    v = ref.bf16_bits_to_f64(allb)
    for b in range(65536):
        bv = brute.bf16_value(b)
        if math.isnan(bv):
            assert math.isnan(v[b])
        else:
            assert v[b] == bv, hex(b)


def test_bf16_round_trip_and_midpoints_exhaustive():
    allb = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    v = ref.bf16_bits_to_f64(allb)
    finite = np.isfinite(v)
    # every finite pattern rounds to itself (zero signs included)
    assert np.array_equal(ref.f64_to_bf16_bits(v[finite]), allb[finite])
    # midpoints between consecutive positive finite patterns go to the even one
    pos = np.arange(0, 0x7F7F, dtype=np.uint32).astype(np.uint16)
    lo = ref.bf16_bits_to_f64(pos)
    hi = ref.bf16_bits_to_f64(pos + 1)
    mid = (lo + hi) / 2.0  # exact in fp64
    want = np.where(pos % 2 == 0, pos, pos + 1).astype(np.uint16)
    assert np.array_equal(ref.f64_to_bf16_bits(mid), want)
    assert np.array_equal(ref.f64_to_bf16_bits(-mid), want | np.uint16(0x8000))


def test_bf16_round_random_against_exact():
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.standard_normal(3000) * 10.0 ** rng.integers(-42, 38, 3000),
                        rng.standard_normal(500) * 2.0 ** -130])
    got = ref.f64_to_bf16_bits(x)
    for xi, g in zip(x, got):
        assert int(g) == brute.bf16_round(float(xi)), xi


def test_bf16_round_is_nearest():
    # nearest among all finite patterns (brute search), random values in a few binades
    allb = np.arange(0, 0x7F80, dtype=np.uint32).astype(np.uint16)
    vals = ref.bf16_bits_to_f64(allb)
    rng = np.random.default_rng(2)
    x = rng.uniform(0.0, 8.0, 400)
    got = ref.bf16_bits_to_f64(ref.f64_to_bf16_bits(x))
    for xi, gi in zip(x, got):
        best = np.min(np.abs(vals - xi))
        assert abs(gi - xi) == best


# ---------------------------------------------------------------------------
# RoPE (Alg. 3 joint RoPE, Eq. 22)
# ---------------------------------------------------------------------------

def test_rope_position_zero_is_identity():
    v = np.random.default_rng(3).standard_normal((5, 96))
    assert np.array_equal(ref.rope(v, 0, 10000.0), v)


def test_rope_d2_is_plane_rotation_by_pos():
    # d = 2: one pair with frequency base^0 = 1, so e1 turns by exactly `pos` radians
    for pos in (1, 2, 7, 4096):
        out = ref.rope(np.array([1.0, 0.0]), pos, 10000.0)
        assert out[0] == pytest.approx(math.cos(pos), abs=1e-15)
        assert out[1] == pytest.approx(math.sin(pos), abs=1e-15)
        out = ref.rope(np.array([0.0, 1.0]), pos, 10000.0)
        assert out[0] == pytest.approx(-math.sin(pos), abs=1e-15)
        assert out[1] == pytest.approx(math.cos(pos), abs=1e-15)


def test_rope_frequency_ladder():
    # the angle of pair j is pos * base^(-2j/d): check pair j against d = 2 rotations
    d, base, pos = 8, 10000.0, 3
    for j in range(d // 2):
        v = np.zeros(d)
        v[j] = 1.0
        out = ref.rope(v, pos, base)
        th = math.atan2(out[j + d // 2], out[j])
        assert th == pytest.approx(math.remainder(pos * base ** (-2 * j / d), 2 * math.pi), abs=1e-12)
        others = np.delete(out, [j, j + d // 2])
        assert np.all(others == 0.0)


def test_rope_preserves_pair_norms():
    rng = np.random.default_rng(4)
    v = rng.standard_normal((3, 128))
    out = ref.rope(v, 32768, 500000.0)
    n_in = v[:, :64] ** 2 + v[:, 64:] ** 2
    n_out = out[:, :64] ** 2 + out[:, 64:] ** 2
    np.testing.assert_allclose(n_out, n_in, rtol=1e-12)


def test_rope_group_law():
    rng = np.random.default_rng(5)
    v = rng.standard_normal(96)
    np.testing.assert_allclose(ref.rope(ref.rope(v, 100, 1e4), 23, 1e4), ref.rope(v, 123, 1e4),
                               rtol=1e-10, atol=1e-12)


def test_rope_relative_position():
    rng = np.random.default_rng(6)
    q, k = rng.standard_normal(64), rng.standard_normal(64)
    base = ref.rope(q, 40, 1e4) @ ref.rope(k, 17, 1e4)
    for s in (1, 100, 3000):
        assert ref.rope(q, 40 + s, 1e4) @ ref.rope(k, 17 + s, 1e4) == pytest.approx(base, rel=1e-9)


# ---------------------------------------------------------------------------
# softmax and single-query attention (Eq. 25-28)
# ---------------------------------------------------------------------------

def test_softmax_normalised_and_shift_invariant():
    s = np.random.default_rng(7).standard_normal(1000) * 5
    p = ref.softmax(s)
    assert math.fsum(p) == pytest.approx(1.0, abs=1e-14)
    np.testing.assert_allclose(ref.softmax(s + 123.0), p, rtol=1e-12)


def test_attention_one_entry_returns_v():
    rng = np.random.default_rng(8)
    q, k, v = rng.standard_normal(64), rng.standard_normal((1, 64)), rng.standard_normal((1, 64))
    o, p = ref.attention_one_query(q, k, v)
    assert p[0] == 1.0
    assert np.array_equal(o, v[0])


def test_attention_identical_keys_mean_of_v():
    rng = np.random.default_rng(9)
    q = rng.standard_normal(32)
    k = np.tile(rng.standard_normal(32), (50, 1))
    v = rng.standard_normal((50, 32))
    o, _ = ref.attention_one_query(q, k, v)
    np.testing.assert_allclose(o, v.mean(axis=0), rtol=1e-12, atol=1e-14)


def test_attention_linear_in_v_and_permutation_invariant():
    rng = np.random.default_rng(10)
    q, k = rng.standard_normal(32), rng.standard_normal((40, 32))
    v1, v2 = rng.standard_normal((40, 32)), rng.standard_normal((40, 32))
    o1, _ = ref.attention_one_query(q, k, v1)
    o2, _ = ref.attention_one_query(q, k, v2)
    o3, _ = ref.attention_one_query(q, k, 2.0 * v1 - 3.0 * v2)
    np.testing.assert_allclose(o3, 2.0 * o1 - 3.0 * o2, rtol=1e-10, atol=1e-12)
    perm = rng.permutation(40)
    o4, _ = ref.attention_one_query(q, k[perm], v1[perm])
    np.testing.assert_allclose(o4, o1, rtol=1e-12, atol=1e-14)


def test_attention_scale_is_inverse_sqrt_d():
    # two keys whose dot products with q differ by sqrt(d) * ln 3: weights 3/4 and 1/4
    d = 16
    q = np.zeros(d)
    q[0] = 1.0
    k = np.zeros((2, d))
    k[0, 0] = math.sqrt(d) * math.log(3.0)
    v = np.array([[1.0] * d, [0.0] * d])
    o, p = ref.attention_one_query(q, k, v)
    assert p[0] == pytest.approx(0.75, rel=1e-14)
    assert p[1] == pytest.approx(0.25, rel=1e-14)


# ---------------------------------------------------------------------------
# RMSNorm, SiLU, MLP
# ---------------------------------------------------------------------------

def test_rms_norm_closed_form_and_scale_law():
    rng = np.random.default_rng(11)
    x = rng.standard_normal(3072)
    eps = 1e-5
    h = ref.rms_norm(x, np.ones_like(x), eps)
    ms = np.mean(x * x)
    assert math.sqrt(np.mean(h * h)) == pytest.approx(math.sqrt(ms / (ms + eps)), rel=1e-12)
    # with eps = 0 the result does not depend on the scale of x
    np.testing.assert_allclose(ref.rms_norm(7.5 * x, np.ones_like(x), 0.0),
                               ref.rms_norm(x, np.ones_like(x), 0.0), rtol=1e-13)
    g = rng.standard_normal(3072)
    np.testing.assert_allclose(ref.rms_norm(x, g, eps), h * g, rtol=1e-13)
    # a constant vector c*1 normalises to c / sqrt(c^2 + eps)
    c = 0.3
    hc = ref.rms_norm(np.full(8, c), np.ones(8), eps)
    np.testing.assert_allclose(hc, c / math.sqrt(c * c + eps), rtol=1e-14)


def test_silu_identities():
    assert ref.silu(np.array([0.0]))[0] == 0.0
    z = np.linspace(-20, 20, 401)
    np.testing.assert_allclose(ref.silu(-z), ref.silu(z) - z, atol=1e-12)
    assert ref.silu(np.array([40.0]))[0] == pytest.approx(40.0, rel=1e-15)
    assert ref.silu(np.array([1.0]))[0] == pytest.approx(1.0 / (1.0 + math.exp(-1.0)), rel=1e-15)


def test_mlp_zero_up_is_zero():
    rng = np.random.default_rng(12)
    h = rng.standard_normal(16)
    out, g, u, a = ref.mlp(h, rng.standard_normal((24, 16)), np.zeros((24, 16)), rng.standard_normal((16, 24)))
    assert np.all(a == 0.0) and np.all(out == 0.0)


@pytest.mark.parametrize("tile", [1, 4, 16, 7, 688])
def test_mlp_interlaced_equals_plain(tile):
    rng = np.random.default_rng(13)
    D, K = 64, 688
    h = rng.standard_normal(D)
    wg, wu, wd = rng.standard_normal((K, D)), rng.standard_normal((K, D)), rng.standard_normal((D, K))
    plain, _, _, a = ref.mlp(h, wg, wu, wd)
    w_gu = formulations.interlace_gate_up(wg, wu, tile)
    assert w_gu.shape == (2 * K, D)
    fused, h_sm = formulations.mlp_interlaced(h, w_gu, wd, tile)
    np.testing.assert_allclose(h_sm, a, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(fused, plain, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(formulations.mlp_alg2(h, wg, wu, wd), plain, rtol=1e-12, atol=1e-12)


def test_interlace_layout_blocks():
    wg = np.arange(6 * 2).reshape(6, 2) + 1000
    wu = np.arange(6 * 2).reshape(6, 2) + 2000
    w = formulations.interlace_gate_up(wg, wu, 2)
    assert np.array_equal(w[0:2], wg[0:2]) and np.array_equal(w[2:4], wu[0:2])
    assert np.array_equal(w[4:6], wg[2:4]) and np.array_equal(w[10:12], wu[4:6])


# ---------------------------------------------------------------------------
# GKVC (Eq. 1)
# ---------------------------------------------------------------------------

def test_gkvc_offset_matches_row_major_index():
    B, G, N, d = 3, 4, 37, 8
    for b in range(B):
        for g in range(G):
            for p in (0, 1, 17, N - 1):
                assert ref.gkvc_offset(b, g, p, G, N, d) == np.ravel_multi_index((b, g, p, 0), (B, G, N, d))


def test_gkvc_append_equals_concat_and_touches_one_slot():
    rng = np.random.default_rng(14)
    B, G, N, d = 2, 3, 10, 4
    cache = rng.integers(0, 65535, (B, G, N, d)).astype(np.uint16)
    new = rng.integers(0, 65535, (B, G, d)).astype(np.uint16)
    pos = np.array([4, 9])
    out = ref.gkvc_append(cache, pos, new)
    for b in range(B):
        p = pos[b]
        cat = np.concatenate([cache[b, :, :p], new[b][:, None, :]], axis=1)
        assert np.array_equal(out[b, :, :p + 1], cat)
        assert np.array_equal(out[b, :, p + 1:], cache[b, :, p + 1:])
    assert np.array_equal(cache, cache)  # input untouched (copy semantics)
    with pytest.raises(ValueError):
        ref.gkvc_append(cache, np.array([4, N]), new)


# ---------------------------------------------------------------------------
# whole layer: brute force, fused == unfused
# ---------------------------------------------------------------------------

BRUTE_CASES = [
    dict(pos=(5,)),
    dict(pos=(0,)),
    dict(pos=(3,), n_kv_heads=2),
    dict(pos=(2, 6), n_kv_heads=2),
    dict(pos=(4,), n_heads=4, n_kv_heads=2, head_dim=2, hidden=8, intermediate=5),
    dict(pos=(7,), base=500000.0, index=101),
]


@pytest.mark.parametrize("case", BRUTE_CASES)
def test_layer_matches_brute_force(case):
    cfg = tiny_cfg(**case)
    inp = inputs.make_layer_inputs(cfg)
    r = run_ref(cfg, inp)
    b = run_brute(cfg, inp)
    for key in ("h1", "a", "y"):
        np.testing.assert_allclose(r[key], np.array(b[key]), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(r["q_rope"], np.array(b["q_rope"]), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(r["o"], np.array(b["o"]), rtol=1e-12, atol=1e-13)
    assert np.array_equal(r["k_new_bits"], np.array(b["k_new_bits"], dtype=np.uint16))
    assert np.array_equal(r["v_new_bits"], np.array(b["v_new_bits"], dtype=np.uint16))
    assert np.array_equal(r["y_bits"], np.array(b["y_bits"], dtype=np.uint16))


def test_layer_pos0_attention_returns_new_v():
    cfg = tiny_cfg(pos=(0,), n_heads=4, n_kv_heads=2)
    inp = inputs.make_layer_inputs(cfg)
    r = run_ref(cfg, inp)
    vnew = ref.bf16_bits_to_f64(r["v_new_bits"][0])
    for h in range(4):
        assert np.array_equal(r["o"][0, h], vnew[h // 2])


@pytest.mark.parametrize("case", [dict(pos=(5,)), dict(pos=(2, 6), n_kv_heads=2),
                                  dict(pos=(31,), hidden=64, n_heads=8, n_kv_heads=2, head_dim=8,
                                       intermediate=100, max_seq=40)])
def test_fused_layer_equals_alg1_alg2(case):
    cfg = tiny_cfg(**case)
    inp = inputs.make_layer_inputs(cfg)
    r = run_ref(cfg, inp)
    y, kcs, vcs = formulations.decode_layer_unfused(
        inp.x, inp.pos, inp.k_cache, inp.v_cache, inp.weights, n_heads=cfg.n_heads,
        n_kv_heads=cfg.n_kv_heads, rope_base=cfg.rope_base, rms_eps=cfg.rms_eps, tile=3)
    np.testing.assert_allclose(y, r["y"], rtol=1e-12, atol=1e-12)
    kc = ref.gkvc_append(inp.k_cache, inp.pos, r["k_new_bits"])
    vc = ref.gkvc_append(inp.v_cache, inp.pos, r["v_new_bits"])
    for b in range(cfg.batch):
        p = int(inp.pos[b])
        assert np.array_equal(kcs[b], kc[b, :, :p + 1])
        assert np.array_equal(vcs[b], vc[b, :, :p + 1])


def test_layer_with_zero_up_projection_returns_h1():
    cfg = tiny_cfg(pos=(3,))
    inp = inputs.make_layer_inputs(cfg)
    inp.weights["w_up"] = np.zeros_like(inp.weights["w_up"])
    r = run_ref(cfg, inp)
    assert np.array_equal(r["y"], r["h1"])


def test_layer_rejects_full_cache():
    cfg = tiny_cfg(pos=(8,))
    inp = inputs.make_layer_inputs(cfg, pos=[7])
    with pytest.raises(ValueError):
        ref.decode_layer_cfg(cfg, inp.x, np.array([8]), inp.k_cache, inp.v_cache, inp.weights)
