"""Parity of the op-by-op baseline (Alg. 1 + Alg. 2, every operator its own
kernel, the Concat rebuilding the cache) with the fp64 oracle, through the C
ABI (MI355X). Same bars as the fused step: untouched cache bytes bit-exact,
the appended K/V within one floored bf16 ulp, y within 2e-2 * max(1, |ref|).
"""
import numpy as np
import pytest

from gpu_harness import check_cache, check_y, log, run_gpu
from oracle import ref
from paper_2607_11211_amd import configs, inputs
from test_gpu_parity import SMALL

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_11211_amd.layer  # noqa: F401  (fails loudly if the library is missing)


CASES = [*SMALL, *(configs.get(n) for n in ("tiny", "phi3_kv1k", "gqa_longctx", "phi3_batch16_ragged"))]


@pytest.mark.parametrize("cfg", CASES, ids=[c.name for c in CASES])
def test_unfused_matches_oracle(cfg):
    log(f"start unfused {cfg.name}")
    inp = inputs.make_layer_inputs(cfg)
    r = ref.decode_layer_cfg(cfg, inp.x, inp.pos, inp.k_cache, inp.v_cache, ref.widen_weights(inp.weights))
    gpu = run_gpu(cfg, inp, unfused=True)
    stats = check_cache(cfg, inp, gpu, r)
    yerr = check_y(gpu, r)
    log(f"unfused {cfg.name}: y_err={yerr:.2e} cache={stats}")


def test_unfused_and_fused_agree_on_phi3_kv4k():
    """Both paths on the same inputs: each within the bar of the oracle, and
    within twice the bar of each other."""
    cfg = configs.get("phi3_kv4k")
    inp = inputs.make_layer_inputs(cfg)
    r = ref.decode_layer_cfg(cfg, inp.x, inp.pos, inp.k_cache, inp.v_cache, ref.widen_weights(inp.weights))
    fused = run_gpu(cfg, inp, debug=False)
    unf = run_gpu(cfg, inp, unfused=True)
    for g in (fused, unf):
        check_cache(cfg, inp, g, r)
        check_y(g, r)
    a, b = ref.bf16_bits_to_f64(fused["y"]), ref.bf16_bits_to_f64(unf["y"])
    assert np.all(np.abs(a - b) <= 4e-2 * np.maximum(1.0, np.abs(r["y"])))
