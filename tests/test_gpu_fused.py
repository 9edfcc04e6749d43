"""The one-kernel decode step (the fused persistent kernel, one sequence)
against the fp64 oracle, through the C ABI (MI355X).

The fused kernel runs the step's six phases in one launch of 256 blocks and
hands data between blocks through agent-coherent stores, loads and per-block
phase flags. The checks are the single-layer bars (untouched cache bytes
bit-exact, appended K/V within one bf16 ulp, y within 2e-2 * max(1, |ref|),
q|k|v, o, h1 and the MLP activation to fp32-level bounds), plus:
  * no bounded wait ran out (the kernel's own count);
  * many steps in a row on one handle (the phase epoch advances) each meet
    the bars, and a rerun of a step gives the same bits;
  * replays of a captured HIP graph (the epoch lives in device memory) equal
    the eager step bit for bit, with eager steps between the replays;
  * the fused step equals the six-kernel step within the bars (not bitwise:
    the merge of the attention splits sums in another order).
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


def phi3(name, index, pos, max_seq):
    return LayerConfig(name=name, index=index, batch=1, hidden=3072, n_heads=32, n_kv_heads=32, head_dim=96,
                       intermediate=8192, rope_base=10000.0, max_seq=max_seq, pos=(pos,))


@pytest.mark.parametrize("cfg", [configs.get("phi3_kv4k"), configs.get("phi3_kv1k"),
                                 phi3("f_pos0", 60, 0, 64), phi3("f_pos63", 61, 63, 128),
                                 phi3("f_pos5000", 62, 5000, 5200)], ids=lambda c: c.name)
def test_fused_matches_oracle(cfg):
    from paper_2607_11211_amd import layer as L
    log(f"start fused {cfg.name}")
    inp = inputs.make_layer_inputs(cfg)
    r = ref.decode_layer_cfg(cfg, inp.x, inp.pos, inp.k_cache, inp.v_cache, inp.weights)
    gpu = run_gpu(cfg, inp, gemm_path=L.GEMM_FUSED, keep=True)
    lay, W = gpu.pop("_layer"), gpu.pop("_weights")
    full_check(cfg, inp, gpu, r)
    assert lay.fused_wait_errors() == 0
    W.free()
    lay.destroy()


def test_fused_consecutive_steps_rerun_and_six_kernel_agreement():
    import torch
    from paper_2607_11211_amd import layer as L
    cfg = phi3("f_steps", 63, 700, 800)
    inp = inputs.make_layer_inputs(cfg)
    lay = L.Layer(cfg)
    lay.set_gemm_path(L.GEMM_FUSED)
    six = L.Layer(cfg)
    six.set_gemm_path(L.GEMM_VECTOR)
    W = lay.pack({k: L.to_device(v) for k, v in inp.weights.items()})
    kc, vc = L.to_device(inp.k_cache), L.to_device(inp.v_cache)
    Wf = ref.widen_weights(inp.weights)
    pos = inp.pos.copy()
    for step in range(6):
        x_bits = inputs.make_x(cfg, seed=300 + step)
        k_before, v_before = L.from_device(kc), L.from_device(vc)
        x = L.to_device(x_bits)
        y = torch.empty_like(x)
        lay.step(W, x, pos, kc, vc, y)
        torch.cuda.synchronize()
        r = ref.decode_layer_cfg(cfg, x_bits, pos, k_before, v_before, Wf)
        step_inp = inputs.LayerInputs(cfg=cfg, x=x_bits, pos=pos.copy(), weights=inp.weights,
                                      k_cache=k_before, v_cache=v_before)
        gpu = {"y": L.from_device(y), "k_cache": L.from_device(kc), "v_cache": L.from_device(vc)}
        full_check(cfg, step_inp, gpu, r, intermediates=False)
        # rerun on the pre-step cache: identical bits
        kc2, vc2 = L.to_device(k_before), L.to_device(v_before)
        y2 = torch.empty_like(x)
        lay.step(W, x, pos, kc2, vc2, y2)
        # the six-kernel step on the same inputs: the same bars, and the same cache slot
        kc3, vc3 = L.to_device(k_before), L.to_device(v_before)
        y3 = torch.empty_like(x)
        six.step(W, x, pos, kc3, vc3, y3)
        torch.cuda.synchronize()
        assert np.array_equal(L.from_device(y2), gpu["y"])
        assert np.array_equal(L.from_device(kc2), gpu["k_cache"])
        g6 = {"y": L.from_device(y3), "k_cache": L.from_device(kc3), "v_cache": L.from_device(vc3)}
        full_check(cfg, step_inp, g6, r, intermediates=False)
        assert np.array_equal(g6["k_cache"], gpu["k_cache"]) and np.array_equal(g6["v_cache"], gpu["v_cache"])
        pos = pos + 1
    assert lay.fused_wait_errors() == 0
    W.free()
    lay.destroy()
    six.destroy()


def test_fused_graph_replays_equal_eager():
    import torch
    from paper_2607_11211_amd import layer as L
    cfg = phi3("f_graph", 64, 2000, 2100)
    inp = inputs.make_layer_inputs(cfg)
    lay = L.Layer(cfg)
    lay.set_gemm_path(L.GEMM_FUSED)
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
        lay.step(W, x, inp.pos, kc, vc, y, stream)  # an eager step between replays
        torch.cuda.synchronize()
        assert np.array_equal(L.from_device(y), y_eager)
    assert lay.fused_wait_errors() == 0
    del g
    W.free()
    lay.destroy()


def test_fused_refuses_other_shapes():
    import torch
    from paper_2607_11211_amd import layer as L
    cfg = configs.get("tiny")
    inp = inputs.make_layer_inputs(cfg)
    lay = L.Layer(cfg)
    lay.set_gemm_path(L.GEMM_FUSED)
    W = lay.pack({k: L.to_device(v) for k, v in inp.weights.items()})
    x = L.to_device(inp.x)
    kc, vc = L.to_device(inp.k_cache), L.to_device(inp.v_cache)
    y = torch.zeros_like(x)
    with pytest.raises(L.FastTPSError) as e:
        lay.step(W, x, inp.pos, kc, vc, y)
    assert e.value.status == L.ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert not L.from_device(y).any()
    W.free()
    lay.destroy()
