"""The allocation-free step (fasttps_decode_step_noalloc) through the C ABI:
its results equal those of fasttps_decode_step on the vector path, bit for
bit, and meet the oracle's bars, on two calls in a row on one handle (the
second smaller, so it runs on what the first left in the static scratch);
a step whose intermediates exceed the static array is refused before any
launch."""
import numpy as np
import pytest

from gpu_harness import check_cache, check_y, log
from oracle import ref
from paper_2607_11211_amd import inputs
from paper_2607_11211_amd.configs import LayerConfig

pytestmark = pytest.mark.gpu

STATIC_BYTES = 8 << 20


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_11211_amd.layer  # noqa: F401  (fails loudly if the library is missing)


def _step(L, lay, W, inp, noalloc):
    import torch
    x = L.to_device(inp.x)
    kc, vc = L.to_device(inp.k_cache), L.to_device(inp.v_cache)
    y = torch.empty_like(x)
    (lay.step_noalloc if noalloc else lay.step)(W, x, inp.pos, kc, vc, y)
    torch.cuda.synchronize()
    return {"y": L.from_device(y), "k_cache": L.from_device(kc), "v_cache": L.from_device(vc)}


def test_noalloc_matches_step_on_two_calls():
    from paper_2607_11211_amd import layer as L
    shape = dict(hidden=1024, n_heads=16, n_kv_heads=4, head_dim=64, intermediate=2816, rope_base=10000.0,
                 max_seq=1100)
    big = LayerConfig(name="na_big", index=61, batch=4, pos=(1099, 512, 77, 1000), **shape)
    small = LayerConfig(name="na_small", index=62, batch=1, pos=(5,), **shape)
    lay = L.Layer(big)
    lay.set_gemm_path(L.GEMM_VECTOR)
    inp_big = inputs.make_layer_inputs(big)
    W = lay.pack({k: L.to_device(v) for k, v in inp_big.weights.items()})
    try:
        for cfg in (big, small):
            inp = inp_big if cfg is big else inputs.LayerInputs(
                cfg=cfg, x=inputs.make_x(cfg), pos=np.asarray(cfg.pos, np.int32), weights=inp_big.weights,
                k_cache=inputs.make_cache(cfg, np.asarray(cfg.pos), "k"),
                v_cache=inputs.make_cache(cfg, np.asarray(cfg.pos), "v"))
            log(f"noalloc {cfg.name}: batch {cfg.batch} pos {list(cfg.pos)}")
            got = _step(L, lay, W, inp, noalloc=True)
            want = _step(L, lay, W, inp, noalloc=False)
            assert np.array_equal(got["y"], want["y"]), "y differs from fasttps_decode_step"
            assert np.array_equal(got["k_cache"], want["k_cache"]) and np.array_equal(got["v_cache"],
                                                                                      want["v_cache"])
            r = ref.decode_layer_cfg(cfg, inp.x, inp.pos, inp.k_cache, inp.v_cache, inp.weights)
            stats = check_cache(cfg, inp, got, r)
            yerr = check_y(got, r)
            log(f"noalloc {cfg.name}: bit-equal to the step; y_err {yerr:.2e} cache {stats}")
    finally:
        W.free()
        lay.destroy()


def test_noalloc_refuses_steps_beyond_its_static_scratch():
    """64 sequences of a hidden-8192, MLP-32768 layer need more than 8 MiB of
    intermediates: refused before any launch, the caches untouched."""
    import torch
    from paper_2607_11211_amd import layer as L
    cfg = LayerConfig(name="na_huge", index=63, batch=64, hidden=8192, n_heads=64, n_kv_heads=16, head_dim=128,
                      intermediate=32768, rope_base=10000.0, max_seq=2, pos=(1,) * 64)
    need = 64 * 4 * ((64 + 32) * 128 + 64 * 128 + 8192 + 32768)
    assert need > STATIC_BYTES
    lay = L.Layer(cfg)
    D, K, q, kv = cfg.hidden, cfg.intermediate, cfg.q_dim, cfg.kv_dim
    raw = {"attn_norm": (D,), "w_q": (q, D), "w_k": (kv, D), "w_v": (kv, D), "w_o": (D, q), "mlp_norm": (D,),
           "w_gate": (K, D), "w_up": (K, D), "w_down": (D, K)}
    W = lay.pack({k: torch.zeros(s, dtype=torch.int16, device="cuda") for k, s in raw.items()})
    try:
        x = torch.zeros((64, D), dtype=torch.int16, device="cuda")
        kc = torch.full((64, cfg.n_kv_heads, 2, 128), 0x1234, dtype=torch.int16, device="cuda")
        vc = kc.clone()
        y = torch.full_like(x, 0x4321)
        with pytest.raises(L.FastTPSError) as e:
            lay.step_noalloc(W, x, cfg.pos, kc, vc, y)
        assert e.value.status == L.ERR_UNSUPPORTED
        assert "static buffer" in str(e.value)
        torch.cuda.synchronize()
        assert bool((kc == 0x1234).all()) and bool((vc == 0x1234).all()) and bool((y == 0x4321).all())
    finally:
        W.free()
        lay.destroy()
