"""The projections on the matrix cores (MFMA, batched decode) against the fp64
oracle, through the C ABI (MI355X).

Both projection paths are forced on the same shapes: the MFMA kernels
(weights in operand-order tiles, activations split into two bf16 levels,
fp32 accumulation) must meet the same bars as the vector GEMVs: untouched
cache bytes bit-exact, appended K/V within one bf16 ulp, y within
2e-2 * max(1, |ref|), and the fp32 intermediates (q|k|v, o, h1, a) within
their bounds. Shapes cover one and two batch tiles, a second and a fourth
grid row (up to the ABI's 64 sequences), ragged positions, matrices whose sizes are not
multiples of the tile (padding of stripes and k-tiles) and the batched and
long-context workloads.
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


SHAPES = [
    # one sequence through the MFMA path (a layer built for two)
    LayerConfig(name="m_b1", index=50, batch=1, hidden=512, n_heads=8, n_kv_heads=2, head_dim=64,
                intermediate=1376, rope_base=10000.0, max_seq=300, pos=(257,)),
    # six sequences: one batch tile, GQA group 4, positions 0 and tile edges
    LayerConfig(name="m_gqa64_b6", index=51, batch=6, hidden=512, n_heads=8, n_kv_heads=2, head_dim=64,
                intermediate=1376, rope_base=10000.0, max_seq=384, pos=(0, 1, 63, 64, 65, 300)),
    # nine sequences: two batch tiles; d = 96; hidden 776 is not a multiple of 32 or 16 (padding)
    LayerConfig(name="m_mha96_b9", index=52, batch=9, hidden=776, n_heads=8, n_kv_heads=8, head_dim=96,
                intermediate=2056, rope_base=10000.0, max_seq=256,
                pos=(127, 200, 255, 3, 17, 64, 100, 128, 150)),
    # twenty sequences: a second grid row of blocks (sequences 16..19)
    LayerConfig(name="m_b20", index=53, batch=20, hidden=256, n_heads=4, n_kv_heads=2, head_dim=64,
                intermediate=688, rope_base=10000.0, max_seq=200,
                pos=tuple(range(0, 200, 10))),
    # hidden 8 against the widest MLP the ABI takes (32768): the down projection's k-tiles padded
    # from 8 inputs and its 32768 inputs in 16 segments (vector) or 1024 k-tiles (MFMA)
    LayerConfig(name="m_longk", index=57, batch=2, hidden=8, n_heads=1, n_kv_heads=1, head_dim=128,
                intermediate=32768, rope_base=10000.0, max_seq=70, pos=(69, 3)),
    # the largest batch the ABI takes (64): four grid rows of MFMA blocks, 16 of vector batch tiles
    LayerConfig(name="m_b64", index=56, batch=64, hidden=256, n_heads=4, n_kv_heads=2, head_dim=64,
                intermediate=688, rope_base=10000.0, max_seq=160,
                pos=tuple((37 * i) % 151 for i in range(64))),
    # d = 128, GQA 4, long RoPE base, intermediate not a multiple of 8 units per stripe boundary
    LayerConfig(name="m_gqa128_b4", index=54, batch=4, hidden=1024, n_heads=8, n_kv_heads=2, head_dim=128,
                intermediate=2824, rope_base=500000.0, max_seq=1100, pos=(5, 511, 1000, 640)),
    # split inputs (operand at least twice a block's weights, 128+ k-tiles): the down projection's
    # 131 k-tiles in 4 parts of 33 (the last 32), one stripe of 16 rows per row group
    LayerConfig(name="m_split_down_b16", index=58, batch=16, hidden=512, n_heads=8, n_kv_heads=2, head_dim=64,
                intermediate=4192, rope_base=10000.0, max_seq=200, pos=tuple((29 * i + 7) % 199 for i in range(16))),
    # split down projection over 33 stripes of 8 rows (hidden 264) and two grid rows (20 sequences)
    LayerConfig(name="m_split_down_b20", index=59, batch=20, hidden=264, n_heads=4, n_kv_heads=4, head_dim=64,
                intermediate=4096, rope_base=10000.0, max_seq=120, pos=tuple((13 * i) % 117 for i in range(20))),
    # split O projection (32 x 128 = 4096 inputs, 16 stripes): its last block writes h1, the gate/up
    # operand and the sums of h1^2
    LayerConfig(name="m_split_o_b12", index=60, batch=12, hidden=256, n_heads=32, n_kv_heads=8, head_dim=128,
                intermediate=688, rope_base=10000.0, max_seq=100, pos=tuple(range(3, 99, 8))),
    # split gate/up projection (4096 inputs, 32 stripes of 8 gate + 8 up rows): RMSNorm2 and SiLU * up
    # in the last block
    LayerConfig(name="m_split_gu_b16", index=61, batch=16, hidden=4096, n_heads=4, n_kv_heads=4, head_dim=64,
                intermediate=256, rope_base=10000.0, max_seq=64, pos=tuple(range(0, 64, 4))),
]


@pytest.mark.parametrize("cfg", SHAPES, ids=lambda c: c.name)
@pytest.mark.parametrize("path", ["matrix", "vector"])
def test_paths_match_oracle(cfg, path):
    from paper_2607_11211_amd import layer as L
    gp = L.GEMM_MATRIX if path == "matrix" else L.GEMM_VECTOR
    log(f"start {cfg.name} {path}")
    inp = inputs.make_layer_inputs(cfg)
    r = ref.decode_layer_cfg(cfg, inp.x, inp.pos, inp.k_cache, inp.v_cache, inp.weights)
    gpu = run_gpu(cfg, inp, gemm_path=gp, max_batch=max(2, cfg.batch))
    full_check(cfg, inp, gpu, r)


@pytest.mark.parametrize("name", ["phi3_batch16_ragged", "gqa_longctx", "phi3_kv1k"])
def test_workloads_matrix_path(name):
    from paper_2607_11211_amd import layer as L
    cfg = configs.get(name)
    log(f"start {name} matrix")
    inp = inputs.make_layer_inputs(cfg)
    cfg = cfg.with_pos(inp.pos)
    r = ref.decode_layer_cfg(cfg, inp.x, inp.pos, inp.k_cache, inp.v_cache, inp.weights)
    gpu = run_gpu(cfg, inp, gemm_path=L.GEMM_MATRIX, max_batch=max(2, cfg.batch))
    full_check(cfg, inp, gpu, r)


def test_batch_changes_on_one_handle():
    """Steps of 16, then 3, then 9 sequences on one handle (the operand
    buffers keep the larger step's rows), each checked against the oracle."""
    import torch
    from paper_2607_11211_amd import layer as L
    big = LayerConfig(name="m_mix", index=55, batch=16, hidden=512, n_heads=8, n_kv_heads=4, head_dim=64,
                      intermediate=1376, rope_base=10000.0, max_seq=160, pos=tuple(range(5, 160, 10)))
    inp = inputs.make_layer_inputs(big)
    lay = L.Layer(big)
    lay.set_gemm_path(L.GEMM_MATRIX)
    W = lay.pack({k: L.to_device(v) for k, v in inp.weights.items()})
    Wf = ref.widen_weights(inp.weights)
    for nb in (16, 3, 9):
        cfg = LayerConfig(name=f"m_mix{nb}", index=55, batch=nb, hidden=512, n_heads=8, n_kv_heads=4,
                          head_dim=64, intermediate=1376, rope_base=10000.0, max_seq=160, pos=big.pos[:nb])
        x_bits = inputs.make_x(cfg, seed=200 + nb)
        kc_h, vc_h = inp.k_cache[:nb].copy(), inp.v_cache[:nb].copy()
        step_inp = inputs.LayerInputs(cfg=cfg, x=x_bits, pos=inp.pos[:nb].copy(), weights=inp.weights,
                                      k_cache=kc_h, v_cache=vc_h)
        r = ref.decode_layer_cfg(cfg, x_bits, step_inp.pos, kc_h, vc_h, Wf)
        gpu = run_gpu(cfg, step_inp, layer=lay, weights=W)
        full_check(cfg, step_inp, gpu, r)
    # a rerun of the last step gives identical bits
    x = L.to_device(x_bits)
    kc, vc = L.to_device(kc_h), L.to_device(vc_h)
    y = torch.empty_like(x)
    lay.step(W, x, step_inp.pos, kc, vc, y)
    torch.cuda.synchronize()
    assert np.array_equal(L.from_device(y), gpu["y"])
    W.free()
    lay.destroy()


def test_path_hook_errors():
    from paper_2607_11211_amd import layer as L
    cfg = configs.get("tiny")
    one = L.Layer(cfg)  # max_batch 1: no MFMA tiles or operands
    with pytest.raises(L.FastTPSError) as e:
        one.set_gemm_path(L.GEMM_MATRIX)
    assert e.value.status == L.ERR_INVALID_ARG
    with pytest.raises(L.FastTPSError) as e:
        one.set_gemm_path(5)
    assert e.value.status == L.ERR_INVALID_ARG
    one.set_gemm_path(L.GEMM_VECTOR)
    # weights packed for max_batch 1 carry no tiles: a two-sequence layer
    # forced onto the matrix path refuses them before any launch
    inp = inputs.make_layer_inputs(cfg)
    W1 = one.pack({k: L.to_device(v) for k, v in inp.weights.items()})
    two = L.Layer(cfg, max_batch=2)
    two.set_gemm_path(L.GEMM_MATRIX)
    import torch
    x = L.to_device(inp.x)
    kc, vc = L.to_device(inp.k_cache), L.to_device(inp.v_cache)
    y = torch.zeros_like(x)
    with pytest.raises(L.FastTPSError) as e:
        two.step(W1, x, inp.pos, kc, vc, y)
    assert e.value.status == L.ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert not L.from_device(y).any()
    assert np.array_equal(L.from_device(kc), inp.k_cache)
    W1.free()
    one.destroy()
    two.destroy()


def test_split_graph_replays_equal_eager():
    """The split projections' tickets are left at zero by every launch: graph
    replays and eager steps in between give the first eager step's bits."""
    import torch
    from paper_2607_11211_amd import layer as L
    cfg = next(c for c in SHAPES if c.name == "m_split_down_b16")
    inp = inputs.make_layer_inputs(cfg)
    lay = L.Layer(cfg)
    lay.set_gemm_path(L.GEMM_MATRIX)
    W = lay.pack({k: L.to_device(v) for k, v in inp.weights.items()})
    x = L.to_device(inp.x)
    kc, vc = L.to_device(inp.k_cache), L.to_device(inp.v_cache)
    y = torch.empty_like(x)
    stream = torch.cuda.current_stream()
    lay.step(W, x, inp.pos, kc, vc, y, stream)
    torch.cuda.synchronize()
    y_eager = L.from_device(y)
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(stream)
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            lay.step(W, x, inp.pos, kc, vc, y, s)
    stream.wait_stream(s)
    torch.cuda.synchronize()
    for rep in range(4):
        y.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(L.from_device(y), y_eager), f"replay {rep} differs from the eager step"
        lay.step(W, x, inp.pos, kc, vc, y, stream)
        torch.cuda.synchronize()
        assert np.array_equal(L.from_device(y), y_eager)
    del g
    W.free()
    lay.destroy()


def test_tiles_only_layout():
    """Weights packed in the MFMA tile order only: steps of one and three
    sequences run the matrix path, meet the oracle's bars and give the bits of
    the matrix path over weights that carry both layouts; steps that need the
    row-major weights are refused before any launch."""
    import torch
    from paper_2607_11211_amd import layer as L
    big = LayerConfig(name="m_tiles", index=62, batch=3, hidden=512, n_heads=8, n_kv_heads=2, head_dim=64,
                      intermediate=1376, rope_base=10000.0, max_seq=160, pos=(5, 77, 150))
    inp = inputs.make_layer_inputs(big)
    dev_w = {k: L.to_device(v) for k, v in inp.weights.items()}
    both = L.Layer(big, max_batch=4)
    both.set_gemm_path(L.GEMM_MATRIX)
    Wb = both.pack(dev_w)
    tl = L.Layer(big, max_batch=4)
    tl.set_weight_layout(L.WEIGHTS_TILES)
    Wt = tl.pack(dev_w)
    Wf = ref.widen_weights(inp.weights)
    for nb in (1, 3):
        cfg = LayerConfig(name=f"m_tiles{nb}", index=62, batch=nb, hidden=512, n_heads=8, n_kv_heads=2,
                          head_dim=64, intermediate=1376, rope_base=10000.0, max_seq=160, pos=big.pos[:nb])
        step_inp = inputs.LayerInputs(cfg=cfg, x=inp.x[:nb].copy(), pos=inp.pos[:nb].copy(), weights=inp.weights,
                                      k_cache=inp.k_cache[:nb].copy(), v_cache=inp.v_cache[:nb].copy())
        r = ref.decode_layer_cfg(cfg, step_inp.x, step_inp.pos, step_inp.k_cache, step_inp.v_cache, Wf)
        log(f"tiles-only step of {nb}")
        gt = run_gpu(cfg, step_inp, layer=tl, weights=Wt)
        full_check(cfg, step_inp, gt, r)
        gb = run_gpu(cfg, step_inp, layer=both, weights=Wb)
        assert np.array_equal(gt["y"], gb["y"])
    # steps that need the row-major weights
    x = L.to_device(inp.x)
    kc, vc = L.to_device(inp.k_cache), L.to_device(inp.v_cache)
    y = torch.zeros_like(x)
    for path in (L.GEMM_VECTOR, L.GEMM_FUSED):
        tl.set_gemm_path(path)
        with pytest.raises(L.FastTPSError) as e:
            tl.step(Wt, x, inp.pos, kc, vc, y)
        assert e.value.status == L.ERR_INVALID_ARG
    tl.set_gemm_path(L.GEMM_AUTO)
    with pytest.raises(L.FastTPSError) as e:
        tl.step_noalloc(Wt, x, inp.pos, kc, vc, y)
    assert e.value.status == L.ERR_INVALID_ARG
    tl.enable_unfused()
    with pytest.raises(L.FastTPSError) as e:
        tl.step_unfused(Wt, x, inp.pos, kc, vc, y)
    assert e.value.status == L.ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert not L.from_device(y).any()
    assert np.array_equal(L.from_device(kc), inp.k_cache) and np.array_equal(L.from_device(vc), inp.v_cache)
    # the fused MLP needs row-major W_down; the layout needs max_batch > 1
    tl.set_mlp_path(L.MLP_FUSED)
    with pytest.raises(L.FastTPSError) as e:
        tl.pack(dev_w)
    assert e.value.status == L.ERR_INVALID_ARG
    one = L.Layer(big, max_batch=1)
    with pytest.raises(L.FastTPSError) as e:
        one.set_weight_layout(L.WEIGHTS_TILES)
    assert e.value.status == L.ERR_INVALID_ARG
    with pytest.raises(L.FastTPSError) as e:
        one.set_weight_layout(7)
    assert e.value.status == L.ERR_INVALID_ARG
    for W in (Wb, Wt):
        W.free()
    for lay in (both, tl, one):
        lay.destroy()


def test_split_and_whole_rows_on_one_handle():
    """Steps of 16 sequences (down projection split across blocks), then 3
    (one batch tile: whole rows), then 16 again on one handle: each checked
    against the oracle, the last with the first step's bits."""
    from paper_2607_11211_amd import layer as L
    big = next(c for c in SHAPES if c.name == "m_split_down_b16")
    inp = inputs.make_layer_inputs(big)
    lay = L.Layer(big)
    lay.set_gemm_path(L.GEMM_MATRIX)
    W = lay.pack({k: L.to_device(v) for k, v in inp.weights.items()})
    Wf = ref.widen_weights(inp.weights)
    ys = []
    for nb in (16, 3, 16):
        cfg = LayerConfig(name=f"m_split_mix{nb}", index=58, batch=nb, hidden=big.hidden, n_heads=big.n_heads,
                          n_kv_heads=big.n_kv_heads, head_dim=big.head_dim, intermediate=big.intermediate,
                          rope_base=big.rope_base, max_seq=big.max_seq, pos=big.pos[:nb])
        step_inp = inputs.LayerInputs(cfg=cfg, x=inp.x[:nb].copy(), pos=inp.pos[:nb].copy(), weights=inp.weights,
                                      k_cache=inp.k_cache[:nb].copy(), v_cache=inp.v_cache[:nb].copy())
        r = ref.decode_layer_cfg(cfg, step_inp.x, step_inp.pos, step_inp.k_cache, step_inp.v_cache, Wf)
        log(f"split/whole-rows step of {nb}")
        gpu = run_gpu(cfg, step_inp, layer=lay, weights=W)
        full_check(cfg, step_inp, gpu, r)
        ys.append(gpu["y"])
    assert np.array_equal(ys[0], ys[2])
    W.free()
    lay.destroy()
