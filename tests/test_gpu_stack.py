"""The 32-layer Phi-3-mini-shaped stack at KV length 4096, one decode step,
through the C ABI (MI355X).

Layer l's output y_l (bf16, the ABI boundary) is layer l+1's input. Two
checks separate per-layer error from compounding:
  * teacher-forced: the oracle's layer l applied to the GPU's own x_l; y_l
    and the appended K/V of every layer meet the single-layer bars, and y_l
    is within one bf16 ulp of the exact value (ulp taken at
    max(|y|, rms(y)/256), as for the appended K/V);
  * free-running: the oracle's own chain x_{l+1} = bf16(y_l). The GPU chain
    must equal it bit for bit until the first layer where a rounding of y
    falls the other way. From there on the two part by the exact stack's own
    sensitivity: with N(0, 0.02) weights each layer's MLP branch is as large
    as its input, so the random 32-layer stack amplifies a one-ulp
    difference by orders of magnitude. That sensitivity is measured with the
    oracle alone: a second oracle chain restarted from the GPU's first
    differing output. The GPU chain's final distance from the free-running
    chain must stay within 4x that chain's (2-norm over the output).
One layer's weights and caches are resident at a time (host and device).
"""
import dataclasses

import numpy as np
import pytest

from gpu_harness import bf16_ulp, check_cache, check_y, log, run_gpu
from oracle import ref
from paper_2607_11211_amd import configs, inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_11211_amd.layer  # noqa: F401  (fails loudly if the library is missing)


def test_stack32_teacher_forced_and_free_running():
    from paper_2607_11211_amd import layer as L
    cfg = configs.get("phi3_stack32_kv4k")
    pos = inputs.make_pos(cfg)
    lay = L.Layer(cfg)
    x_gpu = None      # bf16 bits of the GPU chain's current input
    x_free = None     # bf16 bits of the oracle chain's current input
    x_seed = None     # oracle chain restarted from the GPU's first differing output
    worst_tf = 0.0
    div_gpu, div_seed = [], []
    first_split = None
    try:
        for li in range(cfg.layers):
            inp = inputs.make_layer_inputs(cfg, layer=li, pos=pos)
            if li == 0:
                x_gpu = x_free = inp.x
            inp_gpu = dataclasses.replace(inp, x=x_gpu)
            gpu = run_gpu(cfg, inp_gpu, layer=lay, debug=False)
            W = ref.widen_weights(inp.weights)
            # teacher-forced: the oracle layer on the GPU's own input
            r_tf = ref.decode_layer_cfg(cfg, x_gpu, pos, inp.k_cache, inp.v_cache, W)
            check_cache(cfg, inp_gpu, gpu, r_tf)
            worst_tf = max(worst_tf, check_y(gpu, r_tf))
            y_exact = r_tf["y"]
            rms = np.sqrt(np.mean(y_exact ** 2, axis=-1, keepdims=True))
            ulp = bf16_ulp(np.maximum(np.abs(y_exact), rms / 256.0))
            err = np.abs(ref.bf16_bits_to_f64(gpu["y"]) - y_exact)
            assert np.all(err <= ulp), f"layer {li}: y beyond one ulp, worst err/ulp {float(np.max(err / ulp)):.2f}"
            # free-running: the oracle's own chain (its caches are this layer's)
            r_free = ref.decode_layer_cfg(cfg, x_free, pos, inp.k_cache, inp.v_cache, W)
            if x_seed is not None:
                x_seed = ref.decode_layer_cfg(cfg, x_seed, pos, inp.k_cache, inp.v_cache, W)["y_bits"]
            x_free = r_free["y_bits"]
            x_gpu = gpu["y"]
            if x_seed is None and not np.array_equal(x_gpu, x_free):
                x_seed = x_gpu.copy()
                first_split = li
            yf = ref.bf16_bits_to_f64(x_free)
            div_gpu.append(float(np.max(np.abs(ref.bf16_bits_to_f64(x_gpu) - yf))))
            div_seed.append(float(np.max(np.abs(ref.bf16_bits_to_f64(x_seed) - yf))) if x_seed is not None else 0.0)
            log(f"stack layer {li}: teacher-forced y err {worst_tf:.2e}; max|y_gpu - y_free| {div_gpu[-1]:.3e}; "
                f"max|y_seed - y_free| {div_seed[-1]:.3e}; max|y_free| {float(np.max(np.abs(yf))):.2f}")
            del W, r_tf, gpu, inp, inp_gpu
    finally:
        lay.destroy()
    yf = ref.bf16_bits_to_f64(x_free)
    if first_split is None:
        assert np.array_equal(x_gpu, x_free)
        log("stack32: GPU chain bit-identical to the free-running oracle over all 32 layers")
        return
    d_gpu = float(np.linalg.norm(ref.bf16_bits_to_f64(x_gpu) - yf))
    d_seed = float(np.linalg.norm(ref.bf16_bits_to_f64(x_seed) - yf))
    log(f"stack32: chains bit-identical through layer {first_split - 1}; final |y_gpu - y_free|_2 {d_gpu:.3e}, "
        f"oracle restarted at layer {first_split}: {d_seed:.3e}")
    assert d_gpu <= 4.0 * d_seed, f"GPU chain drifts {d_gpu:.3e} vs the stack's own sensitivity {d_seed:.3e}"
