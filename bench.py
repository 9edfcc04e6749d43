#!/usr/bin/env python3
"""Decode-step benchmark of the FastTPS layer library on one MI355X.

Workload (default): the Phi-3-mini-shaped 32-layer stack, batch 1, KV length
4096 per layer, one decode step = 32 layer steps, each layer with its own
weights and caches (8.9 GB in all, so no layer's data is still in the 256 MB
Infinity Cache when the step comes back to it). The reported value is the
decode-step latency of one layer (step time / 32) in microseconds, next to
the HBM bandwidth it implies over the algorithmic bytes (every weight once
plus the K/V entries read), the dominant kernel's roofline, and the fp64
oracle timed on the host cores.

Inputs are synthetic and seeded: layer 0 comes from the shared input
generator (the bits the oracle sample uses); layers 1..31 are drawn on the
device with the same distributions. Everything is resident in HBM before the
timed region starts.
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
METRIC = "decode-step layer latency (µs) + achieved HBM GB/s vs peak, Phi-3-mini shape"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
ROTATE_BYTES = 2 << 30
WORKLOAD_TEXT = {
    "phi3_stack32_kv4k": "Phi-3-mini-shaped decoder stack, 32 layers, batch 1, KV length 4096 per layer, one decode step",
    "phi3_kv1k": "Phi-3-mini-shaped layer, batch 1, KV length 1024",
    "phi3_kv4k": "Phi-3-mini-shaped layer, batch 1, KV length 4096",
    "phi3_batch16_ragged": "Phi-3-mini-shaped layer, 16 sequences, ragged KV lengths U[512, 4096]",
    "gqa_longctx": "GQA layer (4096 hidden, 32/8 heads x 128, MLP 14336), 4 sequences, KV length 32768",
    "tiny": "tiny layer (256 hidden, 4 x 64 heads, MLP 688), KV length 128",
}


def log(msg: str) -> None:
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def kernel_bytes(cfg, pos, kv_elem_bytes: int = 2, mlp_fused: bool = False):
    """Algorithmic HBM bytes per launch of each kernel (weights once, K/V read
    once; an 8-bit cache reads one byte per element). With the fused MLP the
    slot of the gate/up kernel is the fused kernel (W_gu and W_down) and the
    slot of the down kernel the partial-sum reduction."""
    D, K, d = cfg.hidden, cfg.intermediate, cfg.head_dim
    kv = cfg.kv_read_bytes(pos) * kv_elem_bytes // 2
    return {
        "rmsnorm_qkv": 2 * cfg.qkv_rows * D + 2 * D,
        "attention": kv,
        "attn_combine": 0,
        "oproj_residual": 2 * D * cfg.q_dim,
        "mlp_gate_up": 2 * 2 * K * D + 2 * D + (2 * K * D if mlp_fused else 0),
        "mlp_down": 0 if mlp_fused else 2 * K * D,
        "fused_layer": cfg.weight_bytes() + kv,
    }


# the sources each kernel is built from (a digest of them keys the committed
# counter results to the code they were taken on)
CSRC = "paper_2607_11211_amd/csrc/"
KERNEL_SOURCES = {
    "gemv": [CSRC + "gemv.hip", CSRC + "gemv_body.h", CSRC + "common.h", CSRC + "kernels.h"],
    # the split count (and so the partial-result traffic) is chosen on the host
    "attention": [CSRC + "attention.hip", CSRC + "attn_body.h", CSRC + "common.h", CSRC + "kernels.h",
                  CSRC + "fasttps.cpp"],
    "mfma": [CSRC + "mfma_proj.hip", CSRC + "common.h", CSRC + "kernels.h"],
    # one sequence: the O projection also reads the attention's split records
    # (their count is chosen on the host)
    "gemv_merge": [CSRC + "gemv.hip", CSRC + "gemv_body.h", CSRC + "common.h", CSRC + "kernels.h",
                   CSRC + "fasttps.cpp"],
    "fused": [CSRC + "fused_layer.hip", CSRC + "gemv_body.h", CSRC + "attn_body.h", CSRC + "common.h",
              CSRC + "kernels.h", CSRC + "fasttps.cpp"],
}
KERNEL_GROUP = {"rmsnorm_qkv": "gemv", "oproj_residual": "gemv_merge", "mlp_gate_up": "gemv", "mlp_down": "gemv",
                "attention": "attention", "attn_combine": "attention", "fused_layer": "fused"}


def source_digest(paths) -> str:
    h = hashlib.sha1()
    for p in ([paths] if isinstance(paths, str) else paths):
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def load_traffic(kernel: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the kernel's sources as they are now; else None."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    try:
        info = json.load(open(TRAFFIC_FILE))[kernel]
        if source_digest(info["sources"]) != info["sources_sha1"]:
            return None
        return float(info["bytes_per_launch"])
    except Exception:
        return None


def device_bits(shape, std, mean, gen):
    import torch
    t = torch.randn(shape, generator=gen, device="cuda", dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    if mean != 0.0:
        t.add_(mean)
    return t.to(torch.bfloat16).view(torch.int16)


def device_cache8(cfg, pos, which, fmt, gen):
    """An 8-bit cache of codes drawn on the device (the recipe of inputs.make_cache8:
    finite codes in [0, pos_b), the format's sentinel elsewhere)."""
    import torch
    from paper_2607_11211_amd import inputs
    sentinel = (inputs.K8_SENTINEL if which == "k" else inputs.V8_SENTINEL)[fmt]
    c = torch.full((cfg.batch, cfg.n_kv_heads, cfg.max_seq, cfg.head_dim), sentinel, dtype=torch.uint8, device="cuda")
    for b in range(cfg.batch):
        p = int(pos[b])
        if p <= 0:
            continue
        shape = (cfg.n_kv_heads, p, cfg.head_dim)
        if fmt == "fp8_e4m3":
            r = torch.randint(0, 254, shape, generator=gen, device="cuda", dtype=torch.int16)
            r = torch.where(r < 0x7F, r, r + 1)  # skip the NaN codes 0x7F and 0xFF
        else:
            r = torch.randint(-127, 128, shape, generator=gen, device="cuda", dtype=torch.int16) & 0xFF
        c[b, :, :p].copy_(r.to(torch.uint8))
    return c


def device_layer(cfg, layer, pos, gen, caches=True):
    """Weights and caches of one layer drawn on the device (same recipe as inputs.py)."""
    import torch
    from paper_2607_11211_amd import inputs
    D, K, q, kv = cfg.hidden, cfg.intermediate, cfg.q_dim, cfg.kv_dim
    w = {
        "attn_norm": device_bits((D,), 0.1, 1.0, gen), "w_q": device_bits((q, D), 0.02, 0.0, gen),
        "w_k": device_bits((kv, D), 0.02, 0.0, gen), "w_v": device_bits((kv, D), 0.02, 0.0, gen),
        "w_o": device_bits((D, q), 0.02, 0.0, gen), "mlp_norm": device_bits((D,), 0.1, 1.0, gen),
        "w_gate": device_bits((K, D), 0.02, 0.0, gen), "w_up": device_bits((K, D), 0.02, 0.0, gen),
        "w_down": device_bits((D, K), 0.02, 0.0, gen),
    }
    if not caches:
        return w, None, None
    caches = []
    for sentinel in (inputs.K_SENTINEL, inputs.V_SENTINEL):
        c = torch.full((cfg.batch, cfg.n_kv_heads, cfg.max_seq, cfg.head_dim),
                       int(np.uint16(sentinel).view(np.int16)), dtype=torch.int16, device="cuda")
        for b in range(cfg.batch):
            p = int(pos[b])
            c[b, :, :p].copy_(device_bits((cfg.n_kv_heads, p, cfg.head_dim), 1.0, 0.0, gen))
        caches.append(c)
    return w, caches[0], caches[1]


def cpu_baseline(cfg, seconds: float, kv_fmt: str = "bf16"):
    """The fp64 oracle on a bounded sample: layer 0 of the workload, repeated
    (over the same 8-bit cache as the GPU when kv_fmt names one)."""
    from oracle import ref
    from paper_2607_11211_amd import inputs
    try:
        from threadpoolctl import threadpool_info
        blas = [i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"]
        threads = max(blas) if blas else 1
    except Exception:
        threads = 1
    cores = min(threads, len(os.sched_getaffinity(0)))
    inp = inputs.make_layer_inputs(cfg, layer=0)
    W = ref.widen_weights(inp.weights)   # outside the timer
    kc, vc, kw = inp.k_cache, inp.v_cache, {}
    if kv_fmt != "bf16":
        from oracle import kvquant as kq
        kc = inputs.make_cache8(cfg, inp.pos, "k", kv_fmt)
        vc = inputs.make_cache8(cfg, inp.pos, "v", kv_fmt)
        ks = inputs.make_kv_scales(cfg, "k", kv_fmt)
        vs = inputs.make_kv_scales(cfg, "v", kv_fmt)
        kw = {"kv": kq.KvQuant(kv_fmt, tuple(float(v) for v in ks), tuple(float(v) for v in vs))}
    ref.decode_layer_cfg(cfg, inp.x, inp.pos, kc, vc, W, **kw)  # warm
    reps, t0 = 0, time.perf_counter()
    while True:
        ref.decode_layer_cfg(cfg, inp.x, inp.pos, kc, vc, W, **kw)
        reps += 1
        el = time.perf_counter() - t0
        if (el >= seconds and reps >= 3) or reps >= 100000:
            break
    us = el / reps * 1e6
    # the same sample on one core (BLAS limited to one thread), for a shorter time
    us1, reps1, el1 = None, 0, 0.0
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1, user_api="blas"):
            t0 = time.perf_counter()
            while True:
                ref.decode_layer_cfg(cfg, inp.x, inp.pos, kc, vc, W, **kw)
                reps1 += 1
                el1 = time.perf_counter() - t0
                if (el1 >= seconds / 2 and reps1 >= 2) or reps1 >= 100000:
                    break
        us1 = el1 / reps1 * 1e6
    except Exception:
        us1 = None
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), None)
    except OSError:
        pass
    return {"value": round(us, 1), "unit": "us", "cores": int(cores), "kind": "oracle",
            "sample": f"one layer ({cfg.name} shape, layer 0 inputs"
                      + (f", {kv_fmt} KV cache" if kv_fmt != "bf16" else "")
                      + f"), {reps} repetitions in {el:.1f} s, fp64 numpy, BLAS threads {threads}",
            "gbps": round(kernel_bytes(cfg, cfg.pos, 1 if kv_fmt != "bf16" else 2)["fused_layer"] / us * 1e-3, 2),
            "value_one_core": round(us1, 1) if us1 is not None else None,
            "one_core_sample": f"{reps1} repetitions in {el1:.1f} s, BLAS threads 1" if us1 is not None else None,
            "host_cpus": len(os.sched_getaffinity(0)), "cpu_model": model}


def read_ceiling(nbytes: int = 4 << 30, same_size: int = 0):
    """Measured HBM read rates in the same run: the stream-read probe (16-byte
    loads over 4 GiB, 16 times the Infinity Cache) at a few launch shapes, best
    of three launches each, with plain loads and with the non-temporal policy
    of the weight streams. Returns {flavour: (GB/s, blocks, unroll)}. With
    same_size > 0 also "same_size": the best rate of one non-temporal read
    launch of that many bytes (slices at eight offsets of the 4 GiB buffer, so
    no slice is in the Infinity Cache from the one before), timed like the
    layer's kernels: one launch between two events on its stream, launch and
    ramp included."""
    import ctypes
    import torch
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2607_11211_amd", "libfasttps_probe.so"))
    lib.fasttps_probe_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int,
                                              ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                              ctypes.POINTER(ctypes.c_float)]
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(256, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    best = {}
    for nt, flavour in ((0, "plain"), (1, "nontemporal")):
        for blocks in (2048, 4096, 8192):
            for unroll in (4, 8):
                for _ in range(3):
                    ms = ctypes.c_float()
                    rc = lib.fasttps_probe_stream_read(ctypes.c_void_p(buf.data_ptr()), nbytes,
                                                       ctypes.c_void_p(sink.data_ptr()), blocks, unroll, nt,
                                                       ctypes.c_void_p(stream), ctypes.byref(ms))
                    if rc != 0:
                        raise RuntimeError(f"fasttps_probe_stream_read failed: {rc}")
                    gbps = nbytes / (ms.value * 1e-3) / 1e9
                    if flavour not in best or gbps > best[flavour][0]:
                        best[flavour] = (gbps, blocks, unroll)
    if same_size > 0:
        n = (min(same_size, nbytes // 8) + 15) // 16 * 16
        for blocks in (1024, 2048, 8192):
            for unroll in (1, 2, 4, 8):
                for k in range(8):
                    off = (k * (nbytes // 8)) // 256 * 256
                    ms = ctypes.c_float()
                    rc = lib.fasttps_probe_stream_read(ctypes.c_void_p(buf.data_ptr() + off), n,
                                                       ctypes.c_void_p(sink.data_ptr()), blocks, unroll, 1,
                                                       ctypes.c_void_p(stream), ctypes.byref(ms))
                    if rc != 0:
                        raise RuntimeError(f"fasttps_probe_stream_read failed: {rc}")
                    gbps = n / (ms.value * 1e-3) / 1e9
                    if "same_size" not in best or gbps > best["same_size"][0]:
                        best["same_size"] = (gbps, blocks, unroll)
    del buf
    torch.cuda.empty_cache()
    return best


def sweep(args) -> int:
    """Latency sweeps (the paper's Fig. 6 axes): the fused layer and the op-by-op
    baseline per layer step, over the context length at the Phi-3 shape and
    over the head dimension at the Table 1 shapes (L3.2 d 64, P3 d 96, L2 d 128)
    at 2048 entries. Four rotating layer copies keep the data out of the
    Infinity Cache between visits. One JSON line per point."""
    import torch
    from paper_2607_11211_amd import configs
    from paper_2607_11211_amd import layer as L
    from paper_2607_11211_amd.configs import LayerConfig
    torch.cuda.set_device(0)
    phi3 = dict(hidden=3072, n_heads=32, n_kv_heads=32, head_dim=96, intermediate=8192, rope_base=10000.0)
    points = [("phi3", n, phi3) for n in (512, 1024, 2048, 4096, 8192, 16384, 32768)]
    points += [("llama3.2-1b-like (d 64)", 2048, dict(hidden=2048, n_heads=32, n_kv_heads=32, head_dim=64,
                                                        intermediate=8192, rope_base=10000.0)),
               ("phi3 (d 96)", 2048, phi3),
               ("llama2-7b (d 128)", 2048, dict(hidden=4096, n_heads=32, n_kv_heads=32, head_dim=128,
                                                 intermediate=11008, rope_base=10000.0)),
               ("llama3-8b (GQA 32/8, d 128)", 2048, dict(hidden=4096, n_heads=32, n_kv_heads=8, head_dim=128,
                                                           intermediate=14336, rope_base=500000.0))]
    ncopy = 4
    for name, n, shape in points:
        cfg = LayerConfig(name=f"sweep_{n}", index=40, batch=1, max_seq=n + 64, pos=(n,), **shape)
        pos = np.array([n], dtype=np.int32)
        lay = L.Layer(cfg)
        lay.enable_unfused()
        gen = torch.Generator(device="cuda")
        gen.manual_seed(0xFA57 + n)
        ws, kcs, vcs = [], [], []
        for li in range(ncopy):
            w, kc, vc = device_layer(cfg, li, pos, gen)
            ws.append(lay.pack(w))
            del w
            kcs.append(kc)
            vcs.append(vc)
        x0 = torch.randn((1, cfg.hidden), generator=gen, device="cuda").to(torch.bfloat16).view(torch.int16)
        ys = [torch.empty_like(x0) for _ in range(ncopy)]
        stream = torch.cuda.current_stream()

        def timed(fn):
            fn(stream)
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            s = torch.cuda.Stream()
            s.wait_stream(stream)
            with torch.cuda.stream(s):
                with torch.cuda.graph(g, stream=s):
                    fn(s)
            stream.wait_stream(s)
            torch.cuda.synchronize()
            for _ in range(3):
                g.replay()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(args.steps):
                g.replay()
            e1.record(stream)
            e1.synchronize()
            return e0.elapsed_time(e1) / args.steps * 1e3 / ncopy

        def fused(s):
            for li in range(ncopy):
                lay.step(ws[li], x0, pos, kcs[li], vcs[li], ys[li], s)

        def unfused(s):
            for li in range(ncopy):
                lay.step_unfused(ws[li], x0, pos, kcs[li], vcs[li], ys[li], s)

        us_f, us_u = timed(fused), timed(unfused)
        step_bytes = cfg.step_bytes(pos)
        print(json.dumps({"sweep": name, "kv_entries": n, "d": cfg.head_dim, "us_fused": round(us_f, 2),
                          "us_unfused": round(us_u, 2), "speedup": round(us_u / us_f, 3),
                          "fused_hbm_gbps": round(step_bytes / (us_f * 1e-6) / 1e9, 1),
                          "bytes_per_step": step_bytes}), flush=True)
        for w in ws:
            w.free()
        lay.destroy()
        del kcs, vcs, ys
        torch.cuda.empty_cache()
    return 0


def build_workload(cfg, pos, args, kv: str, gemm: str, log_prefix: str = "", mlp: str = "split"):
    """Resident device copies of a workload: the layers of a stack, or for a
    single layer a chain of independent copies (own weights and caches)
    totalling at least 2 GB (at most 32 copies), so that no copy is still in
    the 256 MB Infinity Cache when the chain comes back to it. Layer 0 comes from the shared input
    generator (the bits the oracle sample uses), the others are drawn on the
    device with the same distributions. Returns a dict of handles and buffers."""
    import torch
    from paper_2607_11211_amd import inputs
    from paper_2607_11211_amd import layer as L
    kv8 = kv != "bf16"
    kb = kernel_bytes(cfg, pos, 1 if kv8 else 2, mlp_fused=mlp == "fused")
    step_bytes = kb["fused_layer"]
    # (a step of a few MB is latency-bound and cached anyway: 32 copies)
    nl = cfg.layers if cfg.layers > 1 else min(max(1, -(-ROTATE_BYTES // step_bytes)), 32)
    log(f"{log_prefix}workload {cfg.name}: {nl} layers, batch {cfg.batch}, pos {pos.tolist()[:4]}")
    gemm_id = {"auto": L.GEMM_AUTO, "vector": L.GEMM_VECTOR, "matrix": L.GEMM_MATRIX, "fused": L.GEMM_FUSED}[gemm]
    lay = L.Layer(cfg, max_batch=max(cfg.batch, 2) if gemm == "matrix" else None)
    lay.set_gemm_path(gemm_id)
    if mlp == "fused":
        lay.set_mlp_path(L.MLP_FUSED)   # before packing: the weights then carry W_down's slices
    weights, kcs, vcs, kss, vss = [], [], [], [], []
    gen = torch.Generator(device="cuda")
    gen.manual_seed(0xFA57 + cfg.index)
    host0 = inputs.make_layer_inputs(cfg, layer=0, pos=pos)
    for li in range(nl):
        if li == 0:
            w = {k: L.to_device(v) for k, v in host0.weights.items()}
            if kv8:
                kc = torch.from_numpy(inputs.make_cache8(cfg, pos, "k", kv)).cuda()
                vc = torch.from_numpy(inputs.make_cache8(cfg, pos, "v", kv)).cuda()
            else:
                kc, vc = L.to_device(host0.k_cache), L.to_device(host0.v_cache)
        else:
            w, kc, vc = device_layer(cfg, li, pos, gen, caches=not kv8)
            if kv8:
                kc = device_cache8(cfg, pos, "k", kv, gen)
                vc = device_cache8(cfg, pos, "v", kv, gen)
        if kv8:
            kss.append(inputs.make_kv_scales(cfg, "k", kv, layer=li))
            vss.append(inputs.make_kv_scales(cfg, "v", kv, layer=li))
        weights.append(lay.pack(w))
        del w
        kcs.append(kc)
        vcs.append(vc)
    x0 = L.to_device(host0.x)
    ys = [torch.empty_like(x0) for _ in range(nl)]
    torch.cuda.synchronize()
    return dict(cfg=cfg, pos=pos, kv=kv, kb=kb, step_bytes=step_bytes, nl=nl, lay=lay, weights=weights, kcs=kcs,
                vcs=vcs, kss=kss, vss=vss, x0=x0, ys=ys)


def free_workload(wl) -> None:
    import torch
    for w in wl["weights"]:
        w.free()
    wl["lay"].destroy()
    wl.clear()
    torch.cuda.empty_cache()


def time_workload(wl, steps: int, warmup: int, graph: bool = True, samples: bool = False):
    """Times one decode step (every layer of the workload once) with stream
    launches and as a HIP-graph replay (checked to reproduce the eager result
    bit for bit on three replays with eager steps in between), and the
    kernels' own durations from events stamped by their dispatches."""
    import torch
    from paper_2607_11211_amd import layer as L
    lay, nl, pos, kv = wl["lay"], wl["nl"], wl["pos"], wl["kv"]
    weights, kcs, vcs, kss, vss, x0, ys = (wl[k] for k in ("weights", "kcs", "vcs", "kss", "vss", "x0", "ys"))
    stream = torch.cuda.current_stream()

    def layer_step(li, x, s_):
        if kv != "bf16":
            lay.step_kv8(weights[li], kv, x, pos, kcs[li], vcs[li], kss[li], vss[li], ys[li], s_)
        else:
            lay.step(weights[li], x, pos, kcs[li], vcs[li], ys[li], s_)

    def step():
        x = x0
        for li in range(nl):
            layer_step(li, x, stream)
            x = ys[li]

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    y_ref = L.from_device(ys[-1])
    out = {}
    # K decode steps launched on the stream
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    e1.synchronize()
    out["stream_ms"] = e0.elapsed_time(e1) / steps
    # per-kernel durations over K more steps (the stamping costs host time per
    # launch, so it stays out of the timed steps above)
    nprof = min(steps * nl, 1 << 16)
    lay.profile_begin(nprof)
    for _ in range(steps):
        step()
    kms = lay.profile_end(nprof)
    names = L.kernel_names()
    out["kern_us"] = {n: float(np.mean(kms[:, i]) * 1e3) for i, n in enumerate(names) if np.any(kms[:, i] > 0)}
    out["graph_ms"] = None
    out["step_samples"] = None
    if graph:
        try:
            g = torch.cuda.CUDAGraph()
            s = torch.cuda.Stream()
            s.wait_stream(stream)
            with torch.cuda.stream(s):
                with torch.cuda.graph(g, stream=s):
                    x = x0
                    for li in range(nl):
                        layer_step(li, x, s)
                        x = ys[li]
            stream.wait_stream(s)
            torch.cuda.synchronize()
            ok = True
            for _ in range(3):  # replays must match the eager result
                g.replay()
                torch.cuda.synchronize()
                ok &= bool(np.array_equal(L.from_device(ys[-1]), y_ref))
                step()
                torch.cuda.synchronize()
            if not ok:
                log("graph replay disagrees with eager steps; graph timing dropped")
            else:
                for _ in range(warmup):
                    g.replay()
                torch.cuda.synchronize()
                e0.record(stream)
                for _ in range(steps):
                    g.replay()
                e1.record(stream)
                e1.synchronize()
                out["graph_ms"] = e0.elapsed_time(e1) / steps
                if samples:
                    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                           for _ in range(steps)]
                    for a0, a1 in evs:
                        a0.record(stream)
                        g.replay()
                        a1.record(stream)
                    torch.cuda.synchronize()
                    out["step_samples"] = np.array([a0.elapsed_time(a1) for a0, a1 in evs])
            del g
        except Exception as ex:  # capture unsupported: report stream timing only
            log(f"graph capture failed: {ex!r}")
    ms = min(out["stream_ms"], out["graph_ms"]) if out["graph_ms"] is not None else out["stream_ms"]
    out["ms_step"] = ms
    out["us_layer"] = ms * 1e3 / nl
    out["gbps"] = wl["step_bytes"] / (out["us_layer"] * 1e-6) / 1e9
    return out


def dominant_roofline(kb, kern_us):
    dominant = max(kern_us, key=kern_us.get)
    ach = kb[dominant] / (kern_us[dominant] * 1e-6) / 1e9 if kb[dominant] else None
    return {"bound": "hbm", "kernel": dominant, "achieved": round(ach, 1) if ach else None,
            "peak": PEAK_HBM_GBPS, "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBPS, 4) if ach else None,
            "traffic": load_traffic(dominant), "algorithmic_bytes": kb[dominant],
            "avg_launch_us": round(kern_us[dominant], 3)}


# the other workloads timed in the default run (each a chain of rotating
# copies; per layer step)
OTHER_WORKLOADS = ("tiny", "phi3_kv1k", "phi3_batch16_ragged", "gqa_longctx")


def other_workloads(args):
    """Per-layer-step figures of the other workloads, measured in the same run
    with a bounded number of steps."""
    from paper_2607_11211_amd import configs, inputs
    res = {}
    for name in OTHER_WORKLOADS:
        cfg = configs.get(name)
        pos = inputs.make_pos(cfg)
        cfg = cfg.with_pos(pos)
        wl = build_workload(cfg, pos, args, "bf16", "auto", log_prefix="  ")
        t = time_workload(wl, steps=max(5, min(args.steps, 20)), warmup=3)
        kb, kern = wl["kb"], t["kern_us"]
        dom = max(kern, key=kern.get)
        entry = {"us_per_layer": round(t["us_layer"], 3),
                 "us_per_layer_graph": round(t["graph_ms"] * 1e3 / wl["nl"], 3) if t["graph_ms"] else None,
                 "us_per_layer_stream": round(t["stream_ms"] * 1e3 / wl["nl"], 3),
                 "bytes_per_layer_step": wl["step_bytes"], "batch": cfg.batch,
                 "kv_entries": [int(p) for p in pos], "rotating_copies": wl["nl"],
                 "kernels_us": {k: round(v, 3) for k, v in kern.items()},
                 "dominant_kernel": dom}
        if name == "tiny":
            entry["note"] = "1.7 MB per step: launch- and latency-bound, no roofline claim"
        else:
            entry["hbm_gbps"] = round(t["gbps"], 1)
            entry["hbm_frac_of_peak"] = round(t["gbps"] / PEAK_HBM_GBPS, 4)
            entry["dominant_kernel_gbps"] = round(kb[dom] / (kern[dom] * 1e-6) / 1e9, 1) if kb[dom] else None
        log(f"  {name}: {entry['us_per_layer']} us per layer step"
            + (f", {entry.get('hbm_gbps')} GB/s" if "hbm_gbps" in entry else "")
            + f"; kernels " + ", ".join(f"{k} {v:.2f}" for k, v in kern.items()))
        res[name] = entry
        free_workload(wl)
    return res


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="phi3_stack32_kv4k")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-graph", action="store_true", help="skip the HIP-graph replay timing")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip timing the other workloads (tiny, Phi-3 at KV 1024, the 16-sequence ragged batch, "
                         "the long-context GQA layer) after the headline one")
    ap.add_argument("--sweep", action="store_true",
                    help="latency sweeps over the context length and the head dimension (fused vs op-by-op), "
                         "one JSON line per point, instead of the benchmark")
    ap.add_argument("--no-unfused", action="store_true",
                    help="skip timing the op-by-op baseline (Alg. 1 + Alg. 2 operators, Concat reloading the cache)")
    ap.add_argument("--gemm", choices=["auto", "vector", "matrix", "fused"], default="auto",
                    help="projection kernels: vector GEMVs (six kernels per step), MFMA (matrix cores), the fused "
                         "one-kernel step (one sequence), or the library's choice")
    ap.add_argument("--batch", type=int, default=None,
                    help="run the workload with this many sequences instead of its own batch (each at the "
                         "workload's KV length, or drawn from a ragged workload's range)")
    ap.add_argument("--mlp", choices=["split", "fused"], default="split",
                    help="MLP kernels: gate/up storing h^sm and a separate down projection (default), or the fused "
                         "MLP keeping h^sm on chip with a partial-sum reduction")
    ap.add_argument("--kv", choices=["bf16", "fp8_e4m3", "int8"], default="bf16",
                    help="KV cache element format: bf16, or 8-bit codes with one scale per KV head "
                         "(fasttps_decode_step_kv8)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="finish with a plain 256 MiB device copy (reference point for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs one decode layer on one GPU; --gpus {args.gpus} is not supported "
              "(sharding across GPUs is not implemented)", file=sys.stderr)
        return 2

    import torch
    from paper_2607_11211_amd import configs, inputs
    from paper_2607_11211_amd import layer as L

    if not torch.cuda.is_available():
        print("bench.py: no GPU", file=sys.stderr)
        return 1
    if args.sweep:
        return sweep(args)
    torch.cuda.set_device(0)
    cfg = configs.get(args.workload)
    text = WORKLOAD_TEXT.get(cfg.name, cfg.name)
    if args.batch is not None:
        if not 1 <= args.batch <= 64:
            print(f"bench.py: --batch {args.batch} is outside 1..64", file=sys.stderr)
            return 2
        cfg = dataclasses.replace(cfg, name=f"{cfg.name}_b{args.batch}", batch=args.batch,
                                  pos=tuple([cfg.pos[0]] * args.batch))
        text += f"; run with {args.batch} sequences"
    pos = inputs.make_pos(cfg)
    cfg = cfg.with_pos(pos)
    kv8 = args.kv != "bf16"
    if kv8:
        if args.gemm == "fused":
            print("bench.py: the one-kernel step reads a bf16 cache only", file=sys.stderr)
            return 2
        text += f"; 8-bit KV cache ({args.kv} codes, one scale per KV head)"

    wl = build_workload(cfg, pos, args, args.kv, args.gemm, mlp=args.mlp)
    nl, kb, step_bytes = wl["nl"], wl["kb"], wl["step_bytes"]
    log(f"resident: {torch.cuda.memory_allocated() / 2**30:.2f} GiB via torch + packed weights")
    t = time_workload(wl, args.steps, args.warmup, graph=not args.no_graph, samples=True)
    stream_ms, graph_ms, kern_us = t["stream_ms"], t["graph_ms"], t["kern_us"]
    if args.mlp == "fused":   # the two MLP slots hold the fused kernel and the reduction
        kb = dict(kb, mlp_fused=kb["mlp_gate_up"], mlp_reduce=kb["mlp_down"])
        kern_us = {{"mlp_gate_up": "mlp_fused", "mlp_down": "mlp_reduce"}.get(k, k): v for k, v in kern_us.items()}
    log(f"stream: {stream_ms:.3f} ms/step, {stream_ms * 1e3 / nl:.2f} us/layer")
    log("kernels (us): " + ", ".join(f"{n} {v:.2f}" for n, v in kern_us.items()))
    if graph_ms is not None:
        log(f"graph: {graph_ms:.3f} ms/step, {graph_ms * 1e3 / nl:.2f} us/layer")
    step_samples = t["step_samples"]

    # the op-by-op baseline on the same workload, replayed as a HIP graph
    unfused = None
    if kv8 and not args.no_unfused:
        log("op-by-op baseline: not built for an 8-bit cache; skipped")
    if not args.no_unfused and not kv8:
        lay, weights, kcs, vcs, x0, ys = (wl[k] for k in ("lay", "weights", "kcs", "vcs", "x0", "ys"))
        stream = torch.cuda.current_stream()
        lay.enable_unfused()
        yu = [torch.empty_like(x0) for _ in range(nl)]

        def step_unfused(s_):
            x = x0
            for li in range(nl):
                lay.step_unfused(weights[li], x, pos, kcs[li], vcs[li], yu[li], s_)
                x = yu[li]

        step_unfused(stream)
        torch.cuda.synchronize()
        gu = torch.cuda.CUDAGraph()
        su = torch.cuda.Stream()
        su.wait_stream(stream)
        with torch.cuda.stream(su):
            with torch.cuda.graph(gu, stream=su):
                step_unfused(su)
        stream.wait_stream(su)
        torch.cuda.synchronize()
        for _ in range(2):
            gu.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            gu.replay()
        e1.record(stream)
        e1.synchronize()
        unf_ms = e0.elapsed_time(e1) / args.steps
        same = bool(np.array_equal(L.from_device(yu[-1]), L.from_device(ys[-1])))
        unfused = {"us_per_layer": round(unf_ms * 1e3 / nl, 3), "ms_per_step": round(unf_ms, 4),
                   "launches_per_layer": 24, "y_bitwise_equal_to_fused": same}
        log(f"unfused baseline (graph): {unf_ms:.3f} ms/step, {unf_ms * 1e3 / nl:.2f} us/layer")
        del gu, yu
    free_workload(wl)

    ms_step, us_layer, gbps = t["ms_step"], t["us_layer"], t["gbps"]
    roofline = dominant_roofline(kb, kern_us)

    dom_bytes = roofline["algorithmic_bytes"] if roofline else 0
    ceil = read_ceiling(same_size=dom_bytes)
    for fl, (g_, b_, u_) in ceil.items():
        what = f"{dom_bytes / 1e6:.1f} MB, one launch" if fl == "same_size" else "4 GiB"
        log(f"read ceiling (stream-read probe, {what}, {fl} loads): {g_:.0f} GB/s at {b_} blocks, unroll {u_}")
    ceiling, c_blocks, c_unroll = ceil["nontemporal"]
    if roofline and roofline.get("achieved") and "same_size" in ceil:
        roofline["frac_of_same_size_read"] = round(roofline["achieved"] / ceil["same_size"][0], 4)
    wbytes = cfg.weight_bytes()

    workloads = None
    if not args.no_workloads and args.workload == "phi3_stack32_kv4k" and args.batch is None and not kv8 \
            and args.gemm == "auto" and args.mlp == "split":
        log("other workloads (per layer step, rotating copies, HIP-graph replay)")
        workloads = other_workloads(args)

    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline: timing the fp64 oracle on one layer")
        one = dataclasses.replace(cfg, layers=1)
        cpu = cpu_baseline(one, args.cpu_seconds, args.kv)
        log(f"cpu baseline: {cpu['value']} us/layer on {cpu['cores']} threads")

    out = {
        "metric": METRIC, "value": round(us_layer, 3), "unit": "us", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": False,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "storage": "bf16" if not kv8 else f"bf16 weights, {args.kv} KV cache",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {text}"
                               + ("" if cfg.layers > 1 else f" ({nl} rotating copies)"),
                   "layers": nl, "global_batch": cfg.batch, "seq_len": int(pos.max()) + 1,
                   "parallelism": "single GPU"},
        "gemm_path": args.gemm, "mlp_path": args.mlp, "kv_cache": args.kv,
        "hbm_gbps": round(gbps, 1), "hbm_frac_of_peak": round(gbps / PEAK_HBM_GBPS, 4),
        "read_ceiling": {"gbps": round(ceiling, 1),
                         "method": f"libfasttps_probe stream read of 4 GiB with 16-byte non-temporal loads, best "
                                   f"launch ({c_blocks} blocks x 256 threads, {c_unroll} loads in flight per thread)",
                         "plain_loads_gbps": round(ceil["plain"][0], 1),
                         "layer_frac_of_ceiling": round(gbps / ceiling, 4),
                         "same_size_read": ({"bytes": dom_bytes, "gbps": round(ceil["same_size"][0], 1),
                                             "method": "one non-temporal stream-read launch of the dominant "
                                                       "kernel's algorithmic bytes between two events, best of "
                                                       "8 slices x 12 launch shapes (best "
                                                       f"{ceil['same_size'][1]} blocks, unroll "
                                                       f"{ceil['same_size'][2]})"}
                                            if "same_size" in ceil else None)},
        "weights_only_gbps": round(wbytes / (us_layer * 1e-6) / 1e9, 1),
        "us_per_layer_p10_p50_p90": ([round(float(np.percentile(step_samples, q)) * 1e3 / nl, 3)
                                      for q in (10, 50, 90)] if step_samples is not None else None),
        "bytes_per_layer_step": step_bytes,
        "us_per_layer_stream": round(stream_ms * 1e3 / nl, 3),
        "us_per_layer_graph": round(graph_ms * 1e3 / nl, 3) if graph_ms is not None else None,
        "kernels_us": {k: round(v, 3) for k, v in kern_us.items()},
        "roofline": roofline,
        "unfused_baseline": (dict(unfused, speedup_of_fused=round(unfused["us_per_layer"] / us_layer, 3))
                             if unfused else None),
        "workloads": workloads,
        "cpu_baseline": cpu,
    }
    if args.calibrate_copy:
        # a plain copy of known size: its FETCH_SIZE / WRITE_SIZE counters
        # (256 MiB each way) scale the counters read for the layer kernels
        src = torch.empty(64 << 20, dtype=torch.float32, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        out["calibration_copy_bytes"] = src.numel() * 4
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
