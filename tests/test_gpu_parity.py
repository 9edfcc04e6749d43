"""Parity of the HIP decode layer with the fp64 oracle, through the C ABI (MI355X).

Bars: untouched cache bytes bit-exact; appended K/V within one bf16 ulp
(measured at max(|ref|, rms/256)); y within 2e-2 * max(1, |ref|) per element;
intermediates (pre-RoPE qkv, attention o, h1, MLP a) to fp32-level bounds.
"""
import numpy as np
import pytest

from gpu_harness import full_check, log, run_gpu
from oracle import ref
from paper_2607_11211_amd import configs, inputs
from paper_2607_11211_amd.configs import LayerConfig

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_11211_amd.layer  # noqa: F401  (fails loudly if the library is missing)


SMALL = [
    # GQA group 4, d=64, several sequences: empty cache, tile edges, multi-split
    LayerConfig(name="s_gqa64", index=10, batch=6, hidden=512, n_heads=8, n_kv_heads=2, head_dim=64,
                intermediate=1376, rope_base=10000.0, max_seq=384, pos=(0, 1, 63, 64, 65, 300)),
    # MHA d=96, last slot of the cache, odd tail
    LayerConfig(name="s_mha96", index=11, batch=3, hidden=768, n_heads=8, n_kv_heads=8, head_dim=96,
                intermediate=2048, rope_base=10000.0, max_seq=256, pos=(127, 200, 255)),
    # GQA group 4, d=128, long base, uneven MLP tile
    LayerConfig(name="s_gqa128", index=12, batch=3, hidden=1024, n_heads=8, n_kv_heads=2, head_dim=128,
                intermediate=2824, rope_base=500000.0, max_seq=1100, pos=(5, 511, 1000)),
    # one KV head, long context: 47 splits (past the one-wave combine's 32: the block combine)
    LayerConfig(name="s_kv1_47split", index=14, batch=1, hidden=256, n_heads=4, n_kv_heads=1, head_dim=64,
                intermediate=688, rope_base=10000.0, max_seq=3136, pos=(3000,)),
    # one KV head, longer context: 126 splits (the block combine, 16 groups of 8 splits at d = 64)
    LayerConfig(name="s_kv1_126split", index=15, batch=1, hidden=256, n_heads=4, n_kv_heads=1, head_dim=64,
                intermediate=688, rope_base=10000.0, max_seq=8064, pos=(8001,)),
    # the smallest shapes the ABI takes: hidden 8 (one 16-byte chunk per row), MLP width 8, a
    # one-slot cache (position 0: the step attends only its own new entry)
    LayerConfig(name="s_min", index=16, batch=1, hidden=8, n_heads=1, n_kv_heads=1, head_dim=64,
                intermediate=8, rope_base=10000.0, max_seq=1, pos=(0,)),
    LayerConfig(name="s_min_b3", index=17, batch=3, hidden=8, n_heads=2, n_kv_heads=1, head_dim=64,
                intermediate=8, rope_base=10000.0, max_seq=2, pos=(0, 1, 1)),
    # the two combine kernels at their boundary: 32 splits (one wave) and 33 (a block)
    LayerConfig(name="s_kv1_32split", index=23, batch=2, hidden=256, n_heads=4, n_kv_heads=1, head_dim=64,
                intermediate=688, rope_base=10000.0, max_seq=2112, pos=(2048, 5)),
    LayerConfig(name="s_kv1_33split", index=24, batch=2, hidden=256, n_heads=4, n_kv_heads=1, head_dim=64,
                intermediate=688, rope_base=10000.0, max_seq=2112, pos=(2049, 2048)),
    # the block combine at d = 96 and d = 128 (10 and 8 thread groups per element): 79 splits over
    # two KV heads, and 141 splits on one KV head with two query heads
    LayerConfig(name="s_d96_79split", index=21, batch=1, hidden=256, n_heads=2, n_kv_heads=2, head_dim=96,
                intermediate=688, rope_base=10000.0, max_seq=5056, pos=(5000,)),
    LayerConfig(name="s_d128_141split", index=22, batch=1, hidden=256, n_heads=2, n_kv_heads=1, head_dim=128,
                intermediate=688, rope_base=500000.0, max_seq=9024, pos=(9000,)),
    # a 128K-entry context on one KV head: 256 splits, the most a step takes (every register of the
    # block combine's threads in use)
    LayerConfig(name="s_ctx128k", index=20, batch=1, hidden=256, n_heads=1, n_kv_heads=1, head_dim=64,
                intermediate=688, rope_base=500000.0, max_seq=131136, pos=(131072,)),
    # one sequence: the O projection merges up to 16 splits itself (16 here), past that the
    # combine kernel runs (17)
    LayerConfig(name="s_merge16", index=25, batch=1, hidden=768, n_heads=8, n_kv_heads=8, head_dim=96,
                intermediate=1024, rope_base=10000.0, max_seq=1100, pos=(1024,)),
    LayerConfig(name="s_merge17", index=26, batch=1, hidden=768, n_heads=8, n_kv_heads=8, head_dim=96,
                intermediate=1024, rope_base=10000.0, max_seq=1100, pos=(1040,)),
    # one sequence with inputs wider than the GEMVs' 64 KB LDS stage (the down projection's
    # 20480 fp32 inputs): the unstaged GEMV kernel at one sequence
    LayerConfig(name="s_wide_k", index=27, batch=1, hidden=512, n_heads=8, n_kv_heads=8, head_dim=64,
                intermediate=20480, rope_base=10000.0, max_seq=200, pos=(150,)),
    # group 2, batch 9 (two batch tiles of the projections)
    LayerConfig(name="s_g2_b9", index=13, batch=9, hidden=256, n_heads=4, n_kv_heads=2, head_dim=64,
                intermediate=688, rope_base=10000.0, max_seq=200, pos=(0, 3, 17, 64, 100, 128, 150, 190, 199)),
]


# splits of 8 tiles and more with one or two query heads per KV head take the
# attention's contiguous-load variant (whole-line loads, LDS exchange): every
# head dimension and both group sizes, and a ragged batch
XCH = [LayerConfig(name=f"x_d{d}_g{g}", index=70 + i, batch=1, hidden=512, n_heads=32 * g, n_kv_heads=32,
                   head_dim=d, intermediate=512, rope_base=10000.0, max_seq=8256, pos=(8192,))
       for i, (d, g) in enumerate([(64, 1), (96, 1), (128, 1), (64, 2), (96, 2), (128, 2)])]
XCH.append(LayerConfig(name="x_d96_ragged3", index=76, batch=3, hidden=512, n_heads=32, n_kv_heads=32, head_dim=96,
                       intermediate=512, rope_base=10000.0, max_seq=16064, pos=(16000, 9000, 12345)))


@pytest.mark.parametrize("cfg", XCH, ids=lambda c: c.name)
def test_contiguous_attention_shapes(cfg):
    log(f"start {cfg.name}")
    inp = inputs.make_layer_inputs(cfg)
    r = ref.decode_layer_cfg(cfg, inp.x, inp.pos, inp.k_cache, inp.v_cache, inp.weights)
    gpu = run_gpu(cfg, inp)
    full_check(cfg, inp, gpu, r)


@pytest.mark.parametrize("cfg", SMALL, ids=lambda c: c.name)
def test_small_shapes(cfg):
    log(f"start {cfg.name}")
    inp = inputs.make_layer_inputs(cfg)
    r = ref.decode_layer_cfg(cfg, inp.x, inp.pos, inp.k_cache, inp.v_cache, inp.weights)
    gpu = run_gpu(cfg, inp)
    full_check(cfg, inp, gpu, r)


@pytest.mark.parametrize("name", ["tiny", "phi3_kv1k", "phi3_kv4k", "gqa_longctx", "phi3_batch16_ragged"])
def test_workloads(name):
    cfg = configs.get(name)
    log(f"start {name}")
    inp = inputs.make_layer_inputs(cfg)
    cfg = cfg.with_pos(inp.pos)
    r = ref.decode_layer_cfg(cfg, inp.x, inp.pos, inp.k_cache, inp.v_cache, inp.weights)
    gpu = run_gpu(cfg, inp)
    full_check(cfg, inp, gpu, r)


def test_maximum_shape():
    """The largest shape the ABI takes: hidden 8192, 64 query heads x 128 (GQA group 4), MLP width
    32768, two sequences; both projection paths against one oracle run."""
    from paper_2607_11211_amd import layer as L
    cfg = LayerConfig(name="s_max", index=19, batch=2, hidden=8192, n_heads=64, n_kv_heads=16, head_dim=128,
                      intermediate=32768, rope_base=500000.0, max_seq=130, pos=(129, 40))
    log(f"start {cfg.name}: drawing inputs and running the oracle")
    inp = inputs.make_layer_inputs(cfg)
    r = ref.decode_layer_cfg(cfg, inp.x, inp.pos, inp.k_cache, inp.v_cache, inp.weights)
    for path, name in ((L.GEMM_MATRIX, "matrix"), (L.GEMM_VECTOR, "vector")):
        log(f"{cfg.name}: {name} path")
        gpu = run_gpu(cfg, inp, gemm_path=path, max_batch=2)
        full_check(cfg, inp, gpu, r)


def test_consecutive_steps_and_determinism():
    """Three tokens in a row on one cache (N_p grows by one per step), and a
    rerun of the same step gives identical bits."""
    import torch
    from paper_2607_11211_amd import layer as L
    cfg = LayerConfig(name="s_steps", index=14, batch=2, hidden=512, n_heads=8, n_kv_heads=2, head_dim=64,
                      intermediate=1376, rope_base=10000.0, max_seq=160, pos=(62, 127))
    inp = inputs.make_layer_inputs(cfg)
    lay = L.Layer(cfg)
    W = lay.pack({k: L.to_device(v) for k, v in inp.weights.items()})
    kc, vc = L.to_device(inp.k_cache), L.to_device(inp.v_cache)
    pos = inp.pos.copy()
    Wf = ref.widen_weights(inp.weights)
    for step in range(3):
        x_bits = inputs.make_x(cfg, seed=100 + step)
        k_before = L.from_device(kc)
        v_before = L.from_device(vc)
        x = L.to_device(x_bits)
        y = torch.empty_like(x)
        lay.step(W, x, pos, kc, vc, y)
        torch.cuda.synchronize()
        r = ref.decode_layer_cfg(cfg, x_bits, pos, k_before, v_before, Wf)
        step_inp = inputs.LayerInputs(cfg=cfg, x=x_bits, pos=pos.copy(), weights=inp.weights,
                                      k_cache=k_before, v_cache=v_before)
        gpu = {"y": L.from_device(y), "k_cache": L.from_device(kc), "v_cache": L.from_device(vc)}
        full_check(cfg, step_inp, gpu, r, intermediates=False)
        # rerun on the pre-step cache: bit-identical y and cache
        kc2, vc2 = L.to_device(k_before), L.to_device(v_before)
        y2 = torch.empty_like(x)
        lay.step(W, x, pos, kc2, vc2, y2)
        torch.cuda.synchronize()
        assert np.array_equal(L.from_device(y2), gpu["y"])
        assert np.array_equal(L.from_device(kc2), gpu["k_cache"])
        pos = pos + 1
    lay.destroy()
    W.free()


def test_error_paths_leave_state_untouched():
    import torch
    from paper_2607_11211_amd import layer as L
    cfg = configs.get("tiny")
    inp = inputs.make_layer_inputs(cfg)
    lay = L.Layer(cfg)
    W = lay.pack({k: L.to_device(v) for k, v in inp.weights.items()})
    x = L.to_device(inp.x)
    kc, vc = L.to_device(inp.k_cache), L.to_device(inp.v_cache)
    y = torch.zeros_like(x)
    with pytest.raises(L.FastTPSError) as e:
        lay.step(W, x, [cfg.max_seq], kc, vc, y)
    assert e.value.status == L.ERR_CACHE_FULL
    with pytest.raises(L.FastTPSError) as e:
        lay.step(W, x, [-1], kc, vc, y)
    assert e.value.status == L.ERR_CACHE_FULL
    with pytest.raises(L.FastTPSError) as e:
        lay.step(W, x, [1, 2], kc, vc, y)
    assert e.value.status == L.ERR_INVALID_ARG
    xb = torch.zeros(2 * cfg.hidden + 8, dtype=torch.int16, device="cuda")
    with pytest.raises(L.FastTPSError) as e:
        lay.step(W, xb[1:], [5], kc, vc, y)
    assert e.value.status == L.ERR_ALIGNMENT
    with pytest.raises(L.FastTPSError) as e:
        lay.step(W, x, [5], kc, vc, x)
    assert e.value.status == L.ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert np.array_equal(L.from_device(kc), inp.k_cache)
    assert np.array_equal(L.from_device(vc), inp.v_cache)
    assert not L.from_device(y).any()
    other = LayerConfig(name="o", index=15, batch=1, hidden=512, n_heads=8, n_kv_heads=2, head_dim=64,
                        intermediate=1376, rope_base=10000.0, max_seq=64, pos=(3,))
    lay2 = L.Layer(other)
    with pytest.raises(L.FastTPSError) as e:
        lay2.step(W, x, [5], kc, vc, y)
    assert e.value.status == L.ERR_BAD_HANDLE
    h = lay.handle
    lay.destroy()
    import ctypes
    assert L.LIB.fasttps_layer_destroy(h) == L.ERR_BAD_HANDLE
    W.free()
    lay2.destroy()
