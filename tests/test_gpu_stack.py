"""The 32-layer Phi-3-mini-shaped stack at KV length 4096, one decode step,
through the C ABI (MI355X).

Layer l's output y_l (bf16, the ABI boundary) is layer l+1's input. Two
checks separate per-layer error from compounding:
  * teacher-forced: the oracle's layer l applied to the GPU's own x_l; y_l
    and the appended K/V of every layer meet the single-layer bars, and y_l
    is within one bf16 ulp of the exact value (ulp taken at
    max(|y|, rms(y)/256), as for the appended K/V);
  * free-running: the oracle's own chain x_{l+1} = bf16(y_l). The GPU chain
    equals it bit for bit until the first layer where a rounding of y falls
    the other way; from there on the two part by the exact stack's own
    sensitivity: with N(0, 0.02) weights each layer's MLP branch is as large
    as its input, so the random 32-layer stack amplifies a one-ulp
    difference by orders of magnitude. That sensitivity is measured with the
    oracle alone, on chains that make the same kind of rounding slips as
    the GPU: at every layer, as many elements of the oracle's bf16 output as
    the GPU's output differs in from the teacher-forced oracle (each such
    difference is one ulp, checked above) are moved by one ulp, at random
    elements and in a random direction (three seeded chains). The GPU
    chain's final distance from the free-running chain must stay within 4x
    the largest of theirs (2-norm over the output).
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


def ulp_step(bits: np.ndarray, idx: np.ndarray, up: np.ndarray) -> np.ndarray:
    """bf16 patterns with the elements idx moved one ulp up (up) or down the
    number line (finite, nonzero values of moderate size here)."""
    out = bits.copy()
    flat = out.reshape(-1)
    v = flat[idx].astype(np.int64)
    neg = (v & 0x8000) != 0
    step = np.where(up != neg, 1, -1)
    step = np.where((v & 0x7FFF) == 0, 1, step)  # from a zero: to the smallest subnormal of its sign
    flat[idx] = (v + step).astype(np.uint16)
    return out


def test_stack32_teacher_forced_and_free_running():
    from paper_2607_11211_amd import layer as L
    cfg = configs.get("phi3_stack32_kv4k")
    pos = inputs.make_pos(cfg)
    lay = L.Layer(cfg)
    n_noise = 3
    rng = np.random.default_rng(0x5EED)
    x_gpu = None      # bf16 bits of the GPU chain's current input
    x_free = None     # bf16 bits of the oracle chain's current input
    x_noise = None    # oracle chains with injected one-ulp roundings
    worst_tf = 0.0
    first_split = None
    try:
        for li in range(cfg.layers):
            inp = inputs.make_layer_inputs(cfg, layer=li, pos=pos)
            if li == 0:
                x_gpu = x_free = inp.x
                x_noise = [inp.x.copy() for _ in range(n_noise)]
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
            for k in range(n_noise):
                yk = ref.decode_layer_cfg(cfg, x_noise[k], pos, inp.k_cache, inp.v_cache, W)["y_bits"]
                if n_diff:
                    idx = rng.choice(yk.size, size=n_diff, replace=False)
                    yk = ulp_step(yk, idx, rng.random(n_diff) < 0.5)
                x_noise[k] = yk
            x_gpu = gpu["y"]
            if first_split is None and not np.array_equal(x_gpu, x_free):
                first_split = li
            yf = ref.bf16_bits_to_f64(x_free)
            d_noise = [float(np.max(np.abs(ref.bf16_bits_to_f64(xn) - yf))) for xn in x_noise]
            log(f"stack layer {li}: teacher-forced y err {worst_tf:.2e}; {n_diff} roundings differ; "
                f"max|y_gpu - y_free| {float(np.max(np.abs(ref.bf16_bits_to_f64(x_gpu) - yf))):.3e}; "
                f"noise chains {', '.join(f'{d:.3e}' for d in d_noise)}; max|y_free| {float(np.max(np.abs(yf))):.2f}")
            del W, r_tf, gpu, inp, inp_gpu
    finally:
        lay.destroy()
    yf = ref.bf16_bits_to_f64(x_free)
    if first_split is None:
        assert np.array_equal(x_gpu, x_free)
        log("stack32: GPU chain bit-identical to the free-running oracle over all 32 layers")
        return
    d_gpu = float(np.linalg.norm(ref.bf16_bits_to_f64(x_gpu) - yf))
    d_noise = [float(np.linalg.norm(ref.bf16_bits_to_f64(xn) - yf)) for xn in x_noise]
    log(f"stack32: chains bit-identical through layer {first_split - 1}; final |y_gpu - y_free|_2 {d_gpu:.3e}; "
        f"oracle chains with the same count of one-ulp roundings: {', '.join(f'{d:.3e}' for d in d_noise)}")
    assert d_gpu <= 4.0 * max(d_noise), f"GPU chain drifts {d_gpu:.3e} vs the stack's own sensitivity {max(d_noise):.3e}"
