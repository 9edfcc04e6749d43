"""The 32-layer Phi-3-mini-shaped stack at KV length 4096, one decode step,
through the C ABI (MI355X).

Layer l's output y_l (bf16, the ABI boundary) is layer l+1's input. Two
checks separate per-layer error from compounding:
  * teacher-forced: the oracle's layer l applied to the GPU's own x_l; y_l
    and the appended K/V of every layer meet the single-layer bars (y within
    2e-2 max(1, |ref|) per element, K/V within one bf16 ulp), and y_l is
    within one bf16 ulp of the exact value (ulp taken at max(|y|, rms(y)/256),
    as for the appended K/V);
  * free-running: the oracle's own chain x_{l+1} = bf16(y_l) against the
    GPU's chain. They agree bit for bit until the first layer where a
    rounding of y falls the other way; from there on they part by the exact
    stack's own sensitivity. With N(0, 0.02) weights each layer's MLP branch
    is as large as its input, and oracle-only chains (no GPU involved) show
    that one one-ulp slip anywhere grows into a relative 2-norm distance of
    about 2e-2 and single elements off by up to 0.4 max(1, |y|) after 32
    layers, whether the chain makes 1 or 64 one-ulp slips per layer (two
    seeds each). So no implementation that differs from the oracle in a
    single rounding can hold the final y to a per-element bar; the test
    reports the final per-element error and holds the chain to a fixed
    ceiling on the relative 2-norm distance, 0.05 (2.5 times those
    oracle-only chains), which a GPU layer that leaves the per-layer bars
    cannot meet by chance.
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


L2_CEILING = 0.05  # relative 2-norm distance of the free-running chains after 32 layers


def test_stack32_teacher_forced_and_free_running():
    from paper_2607_11211_amd import layer as L
    cfg = configs.get("phi3_stack32_kv4k")
    pos = inputs.make_pos(cfg)
    lay = L.Layer(cfg)
    x_gpu = None      # bf16 bits of the GPU chain's current input
    x_free = None     # bf16 bits of the oracle chain's current input
    worst_tf = 0.0
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
            n_diff = int(np.sum(gpu["y"] != r_tf["y_bits"]))
            # free-running: the oracle's own chain (its caches are this layer's)
            x_free = ref.decode_layer_cfg(cfg, x_free, pos, inp.k_cache, inp.v_cache, W)["y_bits"]
            x_gpu = gpu["y"]
            if first_split is None and not np.array_equal(x_gpu, x_free):
                first_split = li
            yf, yg = ref.bf16_bits_to_f64(x_free), ref.bf16_bits_to_f64(x_gpu)
            rel = np.abs(yg - yf) / np.maximum(1.0, np.abs(yf))
            log(f"stack layer {li}: teacher-forced y err {worst_tf:.2e}; {n_diff} roundings differ from the "
                f"teacher-forced oracle; free-running max rel {float(rel.max()):.3e} median "
                f"{float(np.median(rel)):.2e} l2rel {float(np.linalg.norm(yg - yf) / np.linalg.norm(yf)):.3e}; "
                f"max|y_free| {float(np.max(np.abs(yf))):.2f}")
            del W, r_tf, gpu, inp, inp_gpu
    finally:
        lay.destroy()
    yf, yg = ref.bf16_bits_to_f64(x_free), ref.bf16_bits_to_f64(x_gpu)
    if first_split is None:
        assert np.array_equal(x_gpu, x_free)
        log("stack32: GPU chain bit-identical to the free-running oracle over all 32 layers")
        return
    rel = np.abs(yg - yf) / np.maximum(1.0, np.abs(yf))
    l2 = float(np.linalg.norm(yg - yf) / np.linalg.norm(yf))
    log(f"stack32: chains bit-identical through layer {first_split - 1}; final y against the free-running "
        f"oracle: max |dy| / max(1, |y|) {float(rel.max()):.3e} (elements within 2e-2: "
        f"{int(np.sum(rel <= 2e-2))} of {rel.size}), median {float(np.median(rel)):.2e}, relative 2-norm "
        f"distance {l2:.3e} (ceiling {L2_CEILING})")
    assert l2 <= L2_CEILING, f"GPU chain drifts {l2:.3e} from the free-running oracle (ceiling {L2_CEILING})"
