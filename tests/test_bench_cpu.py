"""Host logic of bench.py on the CPU: the per-kernel algorithmic bytes add up
to the step's bytes, the committed counter results are used only while the
kernel sources match their digest, the CPU baseline reports the fields the
JSON line carries, and a request for several GPUs is refused."""
import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2607_11211_amd import configs  # noqa: E402

SEPARATE = ("rmsnorm_qkv", "attention", "attn_combine", "oproj_residual", "mlp_gate_up", "mlp_down")


@pytest.mark.parametrize("name", ["tiny", "phi3_kv1k", "phi3_kv4k", "phi3_batch16_ragged", "gqa_longctx"])
def test_kernel_bytes_add_up_to_the_step(name):
    cfg = configs.get(name)
    kb = bench.kernel_bytes(cfg, cfg.pos)
    assert sum(kb[k] for k in SEPARATE) == cfg.step_bytes()
    assert kb["fused_layer"] == cfg.step_bytes()
    assert kb["attn_combine"] == 0


def test_phi3_dominant_kernel_bytes():
    # 2 x 2K x D bf16 weights of the gate/up pairs plus the gain (2D bytes)
    cfg = configs.get("phi3_kv4k")
    assert bench.kernel_bytes(cfg, cfg.pos)["mlp_gate_up"] == 100_669_440
    # weights and both gains once, plus K and V of the 4096 earlier entries
    assert cfg.step_bytes() == 276_836_352


def test_every_launched_kernel_has_its_sources():
    for k in SEPARATE + ("fused_layer",):
        srcs = bench.KERNEL_SOURCES[bench.KERNEL_GROUP[k]]
        for s in srcs:
            assert os.path.exists(os.path.join(ROOT, s)), s


def test_traffic_used_only_while_sources_match(tmp_path, monkeypatch):
    srcs = bench.KERNEL_SOURCES["gemv"]
    good = {"sources": srcs, "sources_sha1": bench.source_digest(srcs), "bytes_per_launch": 123456}
    stale = dict(good, sources_sha1="0" * 40)
    f = tmp_path / "traffic.json"
    f.write_text(json.dumps({"mlp_gate_up": good, "mlp_down": stale}))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    assert bench.load_traffic("mlp_gate_up") == 123456.0
    assert bench.load_traffic("mlp_down") is None
    assert bench.load_traffic("attention") is None
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "missing.json"))
    assert bench.load_traffic("mlp_gate_up") is None


def test_committed_traffic_file_is_well_formed():
    info = json.load(open(bench.TRAFFIC_FILE))
    for k, v in info.items():
        assert k in SEPARATE
        assert v["bytes_per_launch"] == v["read_bytes"] + v["write_bytes"]
        assert v["sources"] == bench.KERNEL_SOURCES[bench.KERNEL_GROUP[k]]
        assert len(v["sources_sha1"]) == 40


def test_cpu_baseline_fields():
    r = bench.cpu_baseline(configs.get("tiny"), 0.2)
    for key in ("value", "unit", "cores", "kind", "sample"):
        assert key in r
    assert r["kind"] == "oracle" and r["unit"] == "us"
    assert r["value"] > 0 and r["cores"] >= 1
    assert r["value_one_core"] is None or r["value_one_core"] > 0


def test_several_gpus_are_refused(monkeypatch, capsys):
    monkeypatch.setattr(sys, "argv", ["bench.py", "--gpus", "2"])
    assert bench.main() == 2
    assert "--gpus 2" in capsys.readouterr().err


def test_kernel_bytes_of_an_8bit_cache():
    cfg = configs.get("phi3_kv4k")
    kb2, kb1 = bench.kernel_bytes(cfg, cfg.pos), bench.kernel_bytes(cfg, cfg.pos, 1)
    assert kb1["attention"] * 2 == kb2["attention"] == cfg.kv_read_bytes()
    assert kb1["fused_layer"] == cfg.weight_bytes() + cfg.kv_read_bytes() // 2
    assert kb1["mlp_gate_up"] == kb2["mlp_gate_up"]


@pytest.mark.parametrize("fmt", ["fp8_e4m3", "int8"])
def test_cpu_baseline_over_an_8bit_cache(fmt):
    r = bench.cpu_baseline(configs.get("tiny"), 0.2, fmt)
    assert r["kind"] == "oracle" and r["value"] > 0
    assert fmt in r["sample"]
