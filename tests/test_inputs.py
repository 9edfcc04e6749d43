"""Seeded input generator: determinism, layout, sentinels (CPU only)."""
import numpy as np
import pytest

from oracle import brute
from paper_2607_11211_amd import configs, inputs


def test_fp32_to_bf16_matches_exact_rounding():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(20000) * 10.0 ** rng.integers(-30, 30, 20000)).astype(np.float32)
    got = inputs.fp32_to_bf16_bits(x)
    for xi, g in zip(x[:3000], got[:3000]):
        assert int(g) == brute.bf16_round(float(xi))
    # ties: 1 + 2^-8 and 1 + 3*2^-8 are exact in fp32
    t = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8)], dtype=np.float32)
    assert inputs.fp32_to_bf16_bits(t).tolist() == [0x3F80, 0x3F82, 0xBF80]


def test_generator_is_deterministic_and_seeded():
    cfg = configs.get("tiny")
    a = inputs.make_layer_inputs(cfg, seed=0)
    b = inputs.make_layer_inputs(cfg, seed=0)
    c = inputs.make_layer_inputs(cfg, seed=1)
    assert np.array_equal(a.x, b.x) and np.array_equal(a.k_cache, b.k_cache)
    for k in inputs.WEIGHT_NAMES:
        assert np.array_equal(a.weights[k], b.weights[k])
    assert not np.array_equal(a.x, c.x)
    assert not np.array_equal(a.weights["w_q"], a.weights["w_k"][: a.weights["w_q"].shape[0]])


def test_generator_chunking_is_thread_independent(monkeypatch):
    w = [inputs.SEED_DOMAIN, 0, 9, 0, 99]
    n = 3 * inputs.CHUNK + 17
    a = inputs._normal_bf16(w, n, 0.02)
    monkeypatch.setattr(inputs, "_threads", lambda: 1)
    b = inputs._normal_bf16(w, n, 0.02)
    assert np.array_equal(a, b)


def test_cache_layout_and_sentinels():
    cfg = configs.get("tiny")
    inp = inputs.make_layer_inputs(cfg)
    p = int(inp.pos[0])
    assert inp.k_cache.shape == (1, cfg.n_kv_heads, cfg.max_seq, cfg.head_dim)
    assert np.all(inp.k_cache[:, :, p:] == inputs.K_SENTINEL)
    assert np.all(inp.v_cache[:, :, p:] == inputs.V_SENTINEL)
    assert not np.any(inp.k_cache[:, :, :p] == inputs.K_SENTINEL)


def test_value_distributions():
    cfg = configs.get("tiny")
    inp = inputs.make_layer_inputs(cfg)
    from oracle.ref import bf16_bits_to_f64
    wq = bf16_bits_to_f64(inp.weights["w_q"])
    assert abs(wq.std() - 0.02) < 0.002 and abs(wq.mean()) < 0.002
    g = bf16_bits_to_f64(inp.weights["attn_norm"])
    assert abs(g.mean() - 1.0) < 0.03 and abs(g.std() - 0.1) < 0.02
    x = bf16_bits_to_f64(inp.x)
    assert abs(x.std() - 1.0) < 0.15


def test_ragged_positions():
    cfg = configs.get("phi3_batch16_ragged")
    pos = inputs.make_pos(cfg)
    assert pos.shape == (16,) and pos.dtype == np.int32
    assert pos.min() >= 512 and pos.max() <= 4096
    assert len(set(pos.tolist())) > 8
    assert np.array_equal(pos, inputs.make_pos(cfg))


def test_config_bytes_match_paper_shapes():
    # projections 2*(9216*3072 + 3072*3072 + 3*8192*3072) plus the two gains 2*2*3072
    t = configs.get("phi3_kv4k")
    assert t.weight_bytes() == 226_492_416 + 12_288
    assert t.kv_read_bytes() == 2 * 2 * 96 * 32 * 4096
    assert t.step_bytes() == 276_824_064 + 12_288
    c5 = configs.get("gqa_longctx")
    assert c5.step_bytes() == 973_078_528 + 16_384
