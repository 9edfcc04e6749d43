"""The fused MLP with h^sm kept on chip (fasttps_set_mlp_path(FASTTPS_MLP_FUSED);
Section 3.2 "Fusion MLP", Alg. 4, Eq. 29-32) against the oracle, through the C
ABI: one sequence and batch tiles of 2 and 4, MLP widths that do and do not
fill the 256 slices evenly, the Phi-3 and GQA workloads; the step is
deterministic, h^sm is not readable, and weights packed without the path are
refused before any launch."""
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
    # K = 688: 256 slices of 3 units (padded to 8)
    LayerConfig(name="mf_tiny_b1", index=80, batch=1, hidden=256, n_heads=4, n_kv_heads=4, head_dim=64,
                intermediate=688, rope_base=10000.0, max_seq=160, pos=(100,)),
    # K = 200 < 256: one unit per slice, fewer slices than CUs
    LayerConfig(name="mf_k200_b3", index=81, batch=3, hidden=512, n_heads=8, n_kv_heads=2, head_dim=64,
                intermediate=200, rope_base=10000.0, max_seq=100, pos=(0, 50, 99)),
    # batch tiles of 4 and 2 and 1 (7 sequences), K = 1376
    LayerConfig(name="mf_b7", index=82, batch=7, hidden=1024, n_heads=16, n_kv_heads=8, head_dim=64,
                intermediate=1376, rope_base=10000.0, max_seq=300, pos=(5, 17, 299, 64, 128, 200, 1)),
    # wide rows: hidden 4096 (six chunks per lane), K = 14336 (56 units per slice)
    LayerConfig(name="mf_wide_b2", index=83, batch=2, hidden=4096, n_heads=32, n_kv_heads=8, head_dim=128,
                intermediate=14336, rope_base=500000.0, max_seq=200, pos=(150, 7)),
]


def run_fused(cfg, inp, **kw):
    from paper_2607_11211_amd import layer as L
    lay = L.Layer(cfg)
    lay.set_mlp_path(L.MLP_FUSED)
    return run_gpu(cfg, inp, layer=lay, mlp_fused=True, **kw), lay


@pytest.mark.parametrize("cfg", SHAPES, ids=lambda c: c.name)
def test_fused_mlp_shapes(cfg):
    log(f"start fused mlp {cfg.name}")
    inp = inputs.make_layer_inputs(cfg)
    r = ref.decode_layer_cfg(cfg, inp.x, inp.pos, inp.k_cache, inp.v_cache, inp.weights)
    gpu, lay = run_fused(cfg, inp)
    assert "a" not in gpu
    full_check(cfg, inp, gpu, r)
    lay.destroy()


@pytest.mark.parametrize("name", ["phi3_kv4k", "gqa_longctx", "phi3_batch16_ragged"])
def test_fused_mlp_workloads(name):
    cfg = configs.get(name)
    log(f"start fused mlp {name}")
    inp = inputs.make_layer_inputs(cfg)
    cfg = cfg.with_pos(inp.pos)
    r = ref.decode_layer_cfg(cfg, inp.x, inp.pos, inp.k_cache, inp.v_cache, inp.weights)
    gpu, lay = run_fused(cfg, inp)
    full_check(cfg, inp, gpu, r)
    lay.destroy()


def test_fused_mlp_deterministic_and_guarded():
    import torch
    from paper_2607_11211_amd import layer as L
    cfg = SHAPES[2]
    inp = inputs.make_layer_inputs(cfg)
    lay = L.Layer(cfg)
    split_w = lay.pack({k: L.to_device(v) for k, v in inp.weights.items()})   # packed before selecting
    lay.set_mlp_path(L.MLP_FUSED)
    W = lay.pack({k: L.to_device(v) for k, v in inp.weights.items()})
    x = L.to_device(inp.x)
    ys = []
    for _ in range(2):
        kc, vc = L.to_device(inp.k_cache), L.to_device(inp.v_cache)
        y = torch.empty_like(x)
        lay.step(W, x, inp.pos, kc, vc, y)
        torch.cuda.synchronize()
        ys.append(L.from_device(y))
    assert np.array_equal(ys[0], ys[1])
    t = torch.empty(cfg.batch, cfg.intermediate, dtype=torch.float32, device="cuda")
    with pytest.raises(L.FastTPSError) as e:
        lay.debug_read(L.DBG_MLP_A, cfg.batch, t)
    assert e.value.status == L.ERR_INVALID_ARG
    kc, vc = L.to_device(inp.k_cache), L.to_device(inp.v_cache)
    y = torch.full_like(x, 0x1357)
    with pytest.raises(L.FastTPSError) as e:
        lay.step(split_w, x, inp.pos, kc, vc, y)
    assert e.value.status == L.ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert bool((y == 0x1357).all())
    # back to the two-kernel MLP on the same handle: both packs work
    lay.set_mlp_path(L.MLP_SPLIT)
    for w in (split_w, W):
        kc, vc = L.to_device(inp.k_cache), L.to_device(inp.v_cache)
        lay.step(w, x, inp.pos, kc, vc, y)
        torch.cuda.synchronize()
    split_w.free()
    W.free()
    lay.destroy()
