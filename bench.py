#!/usr/bin/env python3
"""Benchmark of the MoE layer over a GPU expert cache on one MI355X.

One step = one ft_moe_forward call (routing, hit/miss split, permutation, grouped SwiGLU expert
FFN over the cache-resident experts, gate-weighted combine) on one synthetic layer instance with
its inputs already resident in HBM.  Steps rotate over --layers distinct layer instances, each
with its own slot-pool weights and routing, so a cycle's working set exceeds the 256 MB
Infinity Cache and weights really stream from HBM.

The default workload is the DeepSeek-V3-shaped prefill chunk (T = 8192 tokens, fp8 block-scaled
weights, 102 of 256 routed experts resident plus the shared expert, hot set re-drawn every 1024
tokens), the largest configuration of the metric that fits one GPU; its roofline is the bf16
MFMA peak, since fp8 weights are widened exactly to bf16 for the matrix cores.  Two decode points
(Qwen3-30B-A3B-shaped T = 32, DeepSeek-V3-shaped T = 64) are timed in the same run and reported
under "decode" with their HBM roofline.

Prints ONE JSON line: tokens/s (whole job), ms per step, the dominant kernel's roofline
fraction (algorithmic flops or bytes of one launch / its HIP-event-timed duration on the
library's stream), and the CPU oracle timed on a bounded sample on this host (one thread and
every CPU of the affinity mask).
"""
import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoE-layer tokens/s + achieved HBM GB/s (decode) / MFMA % (prefill), 1 GPU"
HBM_PEAK_GBS = 8000.0
# hipEventDisableSystemFence: a timing-only event whose record skips the system-scope cache
# writeback and invalidate (the elapsed times are read after a full synchronisation)
HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "fp8": 5000.0}


class HipEvents:
    """hipEvent_t handles through the HIP runtime torch already loaded."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so.7")
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self, flags=0):
        ev = ctypes.c_void_p()
        if self.hip.hipEventCreateWithFlags(ctypes.byref(ev), flags) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")
        return ev.value

    def elapsed_ms(self, a, b) -> float:
        ms = ctypes.c_float()
        if self.hip.hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(a), ctypes.c_void_p(b)) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def destroy(self, ev):
        self.hip.hipEventDestroy(ctypes.c_void_p(ev))


def expert_bytes(lay):
    """Bytes of one complete expert (W1, W3, W2 and their scales) and of its W13 part."""
    H, I = lay.hidden, lay.inter
    if lay.w_dtype == 3:       # MXFP4: half a byte per weight, one scale byte per 32
        w13 = I * H + 2 * I * H // 32
        return w13 + H * I // 2 + H * I // 32, w13
    wb = {0: 4, 1: 2, 2: 1}[lay.w_dtype]
    s13 = (2 * I // 128) * (H // 128) * 4 if lay.w_dtype == 2 else 0
    s2 = (H // 128) * (I // 128) * 4 if lay.w_dtype == 2 else 0
    w13 = 2 * I * H * wb + s13
    return w13 + H * I * wb + s2, w13


def algorithmic_work(lay, route, act_quant=0):
    """Bytes the layer must move and flops it must do, from the realised routing.  With fp8
    activations on the matrix-core path the gate/up GEMM reads x and writes h as one-byte codes
    plus one exponent byte per 128 values."""
    import numpy as np
    T, H, I, E, k = lay.tokens, lay.hidden, lay.inter, lay.n_experts, lay.top_k
    xb = 4 if lay.x_dtype == 0 else 2
    hit_off = route.hit_off.cpu().numpy()
    n_hit = int(route.counts[0])
    u_hit = int(np.count_nonzero(np.diff(hit_off)))
    shared = 1 if lay.shared_slot >= 0 else 0
    S, S13 = expert_bytes(lay)
    lists = 6 * T * k * 4 + 2 * (E + 1) * 4 + 16
    layer_bytes = (u_hit + shared) * S + T * H * xb + T * H * 4 + T * E * 4 + E * 4 + lists
    rows = n_hit + shared * T
    hb = 4 if lay.w_dtype == 0 else 2
    gateup_bytes = (u_hit + shared) * S13 + T * H * xb + rows * I * hb
    if act_quant and T >= 256:
        gateup_bytes = (u_hit + shared) * S13 + (T * H + rows * I) * 129 // 128
    flops = rows * 6 * H * I
    return dict(layer_bytes=layer_bytes, gateup_bytes=gateup_bytes, flops=flops,
                gateup_flops=rows * 4 * H * I, u_hit=u_hit, n_hit=n_hit, rows=rows)


def kernel_source_sha(kernel: str) -> str:
    """Hash of the sources a dominant kernel is built from (its traffic figures are tied to it):
    the GEMM's or the GEMV's file plus the shared device and interface headers, and for the GEMM
    the router, whose tile map orders its tiles."""
    import hashlib
    h = hashlib.sha256()
    files = ("gemm.hip", "route.hip", "route_wave.h") if "gemm" in kernel else ("experts.hip", "route_wave.h")
    for name in (*files, "ftmoe_device.h", "ftmoe_internal.h"):
        with open(os.path.join(ROOT, "paper_2608_16157_amd", "csrc", name), "rb") as fh:
            h.update(name.encode() + b"\0" + fh.read())
    return h.hexdigest()[:16]


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def measured_traffic(key: str):
    """HBM bytes per launch of the dominant kernel from the committed counter runs, or None when
    they were taken on other kernel sources (or never)."""
    try:
        with open(TRAFFIC_FILE) as fh:
            rec = json.load(fh).get(key)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_sha") != kernel_source_sha(rec.get("kernel", "")):
        return None
    return rec.get("traffic_bytes")


def calibrate_copy(mib: int, reps: int = 5):
    """A plain elementwise copy kernel (y = 1 * x, fp32) of known size, for scaling the
    FETCH_SIZE / WRITE_SIZE counters to bytes."""
    import torch
    n = mib * (1 << 20) // 4
    x = torch.ones(n, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    for _ in range(reps):
        torch.mul(x, 1.0, out=y)
    torch.cuda.synchronize()
    print(json.dumps({"calibration": "copy", "bytes_read": 4 * n, "bytes_written": 4 * n,
                      "launches": reps}), flush=True)


def ingest_traffic(key, kernel_match, fetch_csv, write_csv, cal_fetch_csv, cal_write_csv, cal_bytes,
                   per_match=None):
    """Per-launch HBM traffic of the kernel whose name contains kernel_match, from rocprofv3
    --pmc FETCH_SIZE and WRITE_SIZE counter CSVs, each scaled by the same counter's reading for
    the copy calibration kernel of cal_bytes read and cal_bytes written; merged into
    profiles/traffic.json under key.  A stage that the library issues as several dispatches
    (the prefill GEMMs run in chunks of workgroups) is one launch: with per_match, the name of a
    kernel dispatched once per layer forward, the counters of kernel_match are summed and divided
    by that kernel's dispatch count."""
    import csv
    cal = "AUnaryFunctor<float, float, float"     # the y = 1 * x copy kernel

    def readings(path, match):
        vals = []
        for r in csv.DictReader(open(path)):
            if match in r["Kernel_Name"]:
                vals.append(float(r["Counter_Value"]))
        if not vals:
            raise SystemExit(f"no dispatch of {match!r} in {path}")
        return vals

    def per_dispatch(path, match):
        vals = readings(path, match)
        if per_match is None or match == cal:
            return sum(vals) / len(vals)
        return sum(vals) / len(readings(path, per_match))

    f_scale = cal_bytes / per_dispatch(cal_fetch_csv, cal)
    w_scale = cal_bytes / per_dispatch(cal_write_csv, cal)
    fetch = per_dispatch(fetch_csv, kernel_match) * f_scale
    write = per_dispatch(write_csv, kernel_match) * w_scale
    try:
        with open(TRAFFIC_FILE) as fh:
            data = json.load(fh)
    except (OSError, ValueError):
        data = {}
    data[key] = {"kernel": kernel_match, "source_sha": kernel_source_sha(kernel_match),
                 "fetch_bytes": round(fetch), "write_bytes": round(write),
                 "traffic_bytes": round(fetch + write),
                 "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4)}
    with open(TRAFFIC_FILE, "w") as fh:
        json.dump(data, fh, indent=1, sort_keys=True)
        fh.write("\n")
    print(json.dumps({key: data[key]}), flush=True)


def _pool_tensors(cfg, E, device):
    """Random expert weights of one layer shape, E experts, in the bank layout."""
    import torch
    import workloads
    g = torch.Generator(device=device)
    g.manual_seed(12345)
    banks = workloads.alloc_banks(E, cfg.hidden, cfg.inter, cfg.w_dtype, device)
    for e in range(E):
        w1, a1 = workloads._weights(g, cfg.inter, cfg.hidden, cfg.w_dtype, device)
        w3, a3 = workloads._weights(g, cfg.inter, cfg.hidden, cfg.w_dtype, device)
        wd, ad = workloads._weights(g, cfg.hidden, cfg.inter, cfg.w_dtype, device)
        workloads.put_expert(banks, e, cfg.inter, cfg.w_dtype, w1, a1, w3, a3, wd, ad)
    return dict(zip(("w13", "w2", "s13", "s2"), banks))


def measure_bandwidths(cfg_name, n_fill, reps):
    """B_P: the fill kernel copying n_fill complete experts from the pinned host pool into
    device slots; B_H: the CPU branch streaming n_fill experts' weights for one token."""
    import torch
    import paper_2608_16157_amd as ftm
    import workloads
    cfg = workloads.CONFIGS[cfg_name]
    E = n_fill
    dev = _pool_tensors(cfg, E, "cuda")
    pool = {n: (t.cpu().pin_memory() if t is not None else None) for n, t in dev.items()}
    for t in dev.values():
        if t is not None:
            t.zero_()
    S, _ = expert_bytes(type("L", (), {"hidden": cfg.hidden, "inter": cfg.inter, "w_dtype": cfg.w_dtype})())
    desc = dict(hidden=cfg.hidden, inter=cfg.inter, n_experts=E, top_k=min(cfg.top_k, E),
                gating=cfg.gating, w_dtype=cfg.w_dtype, x_dtype=cfg.x_dtype, n_slots=E, shared_slot=-1)
    plan = ftm.FillPlanBuffers(n_fill, E)
    plan.fill_expert.copy_(torch.arange(n_fill, dtype=torch.int32))
    plan.fill_slot.copy_(torch.arange(n_fill, dtype=torch.int32))
    plan.counts.copy_(torch.tensor([n_fill, 0, n_fill, 0], dtype=torch.int32))
    ftm.ft_cache_fill(desc, pool, dev, plan, n_fill)
    torch.cuda.synchronize()
    ok = all(torch.equal(dev[n].cpu(), pool[n]) for n in dev if dev[n] is not None)
    hip = HipEvents()
    stream = torch.cuda.current_stream().cuda_stream
    a, b = hip.create(), hip.create()
    hip.hip.hipEventRecord(a, stream)
    for _ in range(reps):
        ftm.ft_cache_fill(desc, pool, dev, plan, n_fill)
    hip.hip.hipEventRecord(b, stream)
    torch.cuda.synchronize()
    t_fill = hip.elapsed_ms(a, b) / 1e3 / reps
    # CPU branch: one token routed to all n_fill experts
    k = n_fill
    desc_c = dict(desc, top_k=k)
    x = (torch.randn(1, cfg.hidden) * 1.0).to(torch.bfloat16 if cfg.x_dtype == 1 else torch.float32)
    ids = torch.arange(k, dtype=torch.int32).reshape(1, k)
    w = torch.full((1, k), 1.0 / k)
    out = torch.empty(1, cfg.hidden)
    lst = torch.arange(k, dtype=torch.int32)
    workers = ftm.ft_cpu_pool_create(0, pin=True)      # one worker per physical core
    ftm.ft_cpu_experts(desc_c, pool, x, 1, ids, w, lst, out, pool=workers)
    t0 = time.perf_counter()
    for _ in range(reps):
        ftm.ft_cpu_experts(desc_c, pool, x, 1, ids, w, lst, out, pool=workers)
    t_cpu = (time.perf_counter() - t0) / reps
    ftm.ft_cpu_pool_destroy(workers)
    print(json.dumps({
        "measurement": "expert transfer (B_P) and host expert-processing (B_H) bandwidths",
        "workload": f"{cfg_name} experts ({S} bytes each), {n_fill} experts per call",
        "b_pcie_gbs": round(n_fill * S / t_fill / 1e9, 2), "fill_ms": round(t_fill * 1e3, 3),
        "fill_copy_exact": ok,
        "b_host_gbs": round(n_fill * S / t_cpu / 1e9, 2), "cpu_ms": round(t_cpu * 1e3, 3),
        "cpu_pool": "one pinned worker per physical core of the affinity mask",
        "affinity_cpus": len(os.sched_getaffinity(0)),
    }), flush=True)


def hybrid_decode(cfg_name, T, steps, warmup, n_slots, b_pcie, b_host, max_fill):
    """Complete decode layer steps over the GPU expert cache and the host: route once, plan,
    fill, GPU evaluation of hits and fills, CPU branch for the rest (a host function on a
    persistent pinned worker pool), exact merge.  Timed twice by wall clock over back-to-back
    steps: enqueued eagerly, and as replays of one captured HIP graph (new inputs copied into its
    fixed buffers before each replay)."""
    import numpy as np
    import torch
    import paper_2608_16157_amd as ftm
    import workloads
    cfg = workloads.CONFIGS[cfg_name]
    E, H = cfg.n_experts, cfg.hidden
    dev_pool = _pool_tensors(cfg, E, "cuda")
    pool = {n: (t.cpu().pin_memory() if t is not None else None) for n, t in dev_pool.items()}
    dev = {n: (torch.zeros((n_slots,) + tuple(t.shape[1:]), dtype=t.dtype, device="cuda")
               if t is not None else None) for n, t in dev_pool.items()}
    del dev_pool
    desc = dict(hidden=H, inter=cfg.inter, n_experts=E, top_k=cfg.top_k, gating=cfg.gating,
                w_dtype=cfg.w_dtype, x_dtype=cfg.x_dtype, n_slots=n_slots, shared_slot=-1)
    workers = ftm.ft_cpu_pool_create(0, pin=True)
    g = torch.Generator(device="cuda")
    g.manual_seed(77)
    rank = torch.randperm(E, generator=g, device="cuda").float() + 1
    bias = -cfg.zipf_s * torch.log(rank)
    n = warmup + steps
    logits = [torch.randn(T, E, generator=g, device="cuda") + bias[None, :] for _ in range(n)]
    xs = [torch.randn(T, H, generator=g, device="cuda").to(torch.bfloat16) for _ in range(n)]
    res = {}
    for mode in ("eager", "graph"):
        table = torch.full((E,), -1, dtype=torch.int32, device="cuda")
        state = ftm.CacheState(torch.full((n_slots,), -1, dtype=torch.int32, device="cuda"),
                               torch.zeros(n_slots, dtype=torch.int32, device="cuda"),
                               torch.zeros(1, dtype=torch.int32, device="cuda"))
        for t in dev.values():
            if t is not None:
                t.zero_()
        route = ftm.RouteBuffers(T, cfg.top_k, E)
        plan = ftm.FillPlanBuffers(max_fill, E)
        ws = ftm.alloc_workspace(desc, T)
        host = ftm.HybridHostBuffers(T, cfg.top_k, E, H, torch.bfloat16)
        out = torch.empty(T, H, dtype=torch.float32, device="cuda")
        lg_buf = torch.empty(T, E, device="cuda")
        x_buf = torch.empty(T, H, dtype=torch.bfloat16, device="cuda")
        counts = torch.zeros(n, 4, dtype=torch.int32, device="cuda")

        def call(i, lg, xx, stream=None):
            ftm.ft_moe_step_hybrid(desc, dev, pool, lg, table, state, b_pcie, b_host, max_fill, i + 1,
                                   xx, T, out, route, plan, host, ws, workers, stream=stream)

        if mode == "graph":
            graph = torch.cuda.CUDAGraph()
            cap = torch.cuda.Stream()
            torch.cuda.synchronize()
            with torch.cuda.graph(graph, stream=cap, capture_error_mode="relaxed"):
                call(0, lg_buf, x_buf, stream=cap)
            torch.cuda.synchronize()
        for i in range(n):
            if i == warmup:
                torch.cuda.synchronize()
                t0 = time.perf_counter()
            if mode == "eager":
                call(i, logits[i], xs[i])
            else:
                lg_buf.copy_(logits[i])
                x_buf.copy_(xs[i])
                graph.replay()
            counts[i].copy_(plan.counts)
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / steps
        c = counts[warmup:].float().mean(0).tolist()
        res[mode] = {"ms_per_step": round(dt * 1e3, 4), "tokens_per_s": round(T / dt, 1),
                     "fills_per_step": round(c[0], 2), "cpu_experts_per_step": round(c[1], 2),
                     "missing_experts_per_step": round(c[2], 2)}
        if mode == "graph":
            del graph
    ftm.ft_cpu_pool_destroy(workers)
    print(json.dumps({
        "measurement": "hybrid decode layer step (GPU expert cache + fills + CPU branch + merge), "
                       "back-to-back steps, wall clock",
        "workload": f"{cfg_name} shapes, T={T}, {n_slots} of {E} experts cacheable, Zipf "
                    f"{cfg.zipf_s} routing, B_P={b_pcie} B_H={b_host} GB/s, K={max_fill}, CPU branch "
                    f"on one pinned worker per CPU of the affinity mask",
        **res}), flush=True)


def cache_plan_timing(cfg_name, T, steps, warmup, n_slots, b_pcie, b_host, max_fill):
    """Device-side cache control alone (ft_route_only then ft_cache_plan, row f1) over decode
    steps whose cache state evolves: HIP events on the library's stream around each call.  The
    host issues one step at a time, so these intervals include the launch gaps; the kernels'
    own durations come from a kernel trace of the same run."""
    import torch
    import paper_2608_16157_amd as ftm
    import workloads
    cfg = workloads.CONFIGS[cfg_name]
    E = cfg.n_experts
    desc = dict(hidden=cfg.hidden, inter=cfg.inter, n_experts=E, top_k=cfg.top_k, gating=cfg.gating,
                w_dtype=cfg.w_dtype, x_dtype=cfg.x_dtype, n_slots=n_slots, shared_slot=-1)
    table = torch.full((E,), -1, dtype=torch.int32, device="cuda")
    state = ftm.CacheState(torch.full((n_slots,), -1, dtype=torch.int32, device="cuda"),
                           torch.zeros(n_slots, dtype=torch.int32, device="cuda"))
    route = ftm.RouteBuffers(T, cfg.top_k, E)
    plan = ftm.FillPlanBuffers(max_fill, E)
    ws = ftm.alloc_workspace(desc, T)
    g = torch.Generator(device="cuda")
    g.manual_seed(78)
    rank = torch.randperm(E, generator=g, device="cuda").float() + 1
    bias = -cfg.zipf_s * torch.log(rank)
    n = warmup + steps
    logits = [torch.randn(T, E, generator=g, device="cuda") + bias[None, :] for _ in range(n)]
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n)]
    counts = []
    for i in range(n):
        e0, e1, e2 = evs[i]
        e0.record()
        ftm.ft_route_only(desc, logits[i], table, T, route, ws)
        e1.record()
        ftm.ft_cache_plan(desc, route, T, table, state, b_pcie, b_host, max_fill, i + 1, plan)
        e2.record()
        if i >= warmup:
            counts.append(plan.counts.clone())
    torch.cuda.synchronize()
    r_us = sum(evs[i][0].elapsed_time(evs[i][1]) for i in range(warmup, n)) * 1e3 / steps
    p_us = sum(evs[i][1].elapsed_time(evs[i][2]) for i in range(warmup, n)) * 1e3 / steps
    c = torch.stack(counts).float().mean(0).tolist()
    print(json.dumps({
        "measurement": "device-side cache control: ft_route_only then ft_cache_plan per decode step",
        "workload": f"{cfg_name} shapes, T={T}, {n_slots} of {E} experts cacheable, Zipf {cfg.zipf_s} "
                    f"routing, B_P={b_pcie} B_H={b_host} GB/s, K={max_fill}, {steps} steps",
        "route_us_with_launch": round(r_us, 2), "cache_plan_us_with_launch": round(p_us, 2),
        "fills_per_step": round(c[0], 2), "cpu_experts_per_step": round(c[1], 2),
        "missing_experts_per_step": round(c[2], 2)}), flush=True)


def prefill_pipeline(cfg_name, T, n_layers, reps):
    """Full-layer double-buffered prefill (ft_prefill_layers): a T-token chunk through n_layers
    MoE layers whose complete expert sets are loaded from pinned host memory, with the loads
    overlapped against the evaluation and serialised, next to the loads alone and the
    evaluation alone (HIP events on the evaluation stream)."""
    import torch
    import paper_2608_16157_amd as ftm
    import workloads
    cfg = workloads.CONFIGS[cfg_name]
    E = cfg.n_experts
    shared = cfg.shared_expert
    n_slots = E + (1 if shared else 0)
    n_pools = min(2, n_layers)           # two distinct layers' expert sets, cycled over the layers
    pools, logits, xs = [], [], []
    for l in range(n_pools):
        lay = workloads.make_layer(cfg_name, T, layer=l, device="cuda", resident_frac=1.0)
        order = lay.slot_table.tolist() + ([lay.shared_slot] if shared else [])
        idx = torch.tensor(order, dtype=torch.long, device="cuda")
        pool = {}
        for n in ("w13", "w2", "s13", "s2"):
            t = getattr(lay, n)
            if t is None:
                pool[n] = None
                continue
            pool[n] = torch.empty(t.shape, dtype=t.dtype, pin_memory=True)
            pool[n].copy_(t.index_select(0, idx))
        pools.append(pool)
        logits.append(lay.logits)
        xs.append(lay.x)
        del lay, idx
        torch.cuda.empty_cache()
    desc = dict(hidden=cfg.hidden, inter=cfg.inter, n_experts=E, top_k=cfg.top_k, gating=cfg.gating,
                w_dtype=cfg.w_dtype, x_dtype=cfg.x_dtype, n_slots=n_slots, shared_slot=E if shared else -1)
    bufs = [{n: (torch.empty(t.shape, dtype=t.dtype, device="cuda") if t is not None else None)
             for n, t in pools[0].items()} for _ in range(2)]
    layer_bytes = sum(t.numel() * t.element_size() for t in pools[0].values() if t is not None)
    table = torch.arange(E, dtype=torch.int32, device="cuda")
    route = ftm.RouteBuffers(T, cfg.top_k, E)
    ws = ftm.alloc_workspace(desc, T)
    outs = [torch.empty(T, cfg.hidden, device="cuda") for _ in range(n_layers)]
    hl = [pools[l % n_pools] for l in range(n_layers)]
    lg = [logits[l % n_pools] for l in range(n_layers)]
    xl = [xs[l % n_pools] for l in range(n_layers)]
    copy_stream = torch.cuda.Stream()
    hip = HipEvents()
    stream = torch.cuda.current_stream().cuda_stream
    a, b = hip.create(), hip.create()

    def timed(fn):
        fn()                                  # warm-up
        torch.cuda.synchronize()
        hip.hip.hipEventRecord(a, stream)
        for _ in range(reps):
            fn()
        hip.hip.hipEventRecord(b, stream)
        torch.cuda.synchronize()
        return hip.elapsed_ms(a, b) / reps / n_layers

    def loads_only():
        for l in range(n_layers):
            for n, t in hl[l].items():
                if t is not None:
                    bufs[l % 2][n].copy_(t, non_blocking=True)

    def compute_only():
        for l in range(n_layers):
            ftm.ft_moe_forward(desc, bufs[l % 2], lg[l], table, xl[l], T, outs[l], route, ws)

    t_overlap = timed(lambda: ftm.ft_prefill_layers(desc, hl, bufs, table, lg, xl, T, outs, route, ws,
                                                    overlap=True, copy_stream=copy_stream))
    t_serial = timed(lambda: ftm.ft_prefill_layers(desc, hl, bufs, table, lg, xl, T, outs, route, ws,
                                                   overlap=False))
    t_load = timed(loads_only)
    t_comp = timed(compute_only)
    print(json.dumps({
        "measurement": "full-layer double-buffered prefill (ft_prefill_layers)",
        "workload": f"{cfg_name} shapes, T={T} tokens, {n_layers} MoE layers, every layer's "
                    f"{n_slots} experts ({layer_bytes} bytes) loaded from pinned host memory, "
                    f"{n_pools} distinct layers' weights cycled",
        "ms_per_layer_overlap": round(t_overlap, 3), "ms_per_layer_serial": round(t_serial, 3),
        "ms_per_layer_loads_only": round(t_load, 3), "ms_per_layer_compute_only": round(t_comp, 3),
        "load_gbs": round(layer_bytes / (t_load / 1e3) / 1e9, 2),
        "tokens_per_s_overlap": round(T / (t_overlap * n_layers / 1e3), 1),
        "tokens_per_s_serial": round(T / (t_serial * n_layers / 1e3), 1),
        "serial_cost_frac": round(1 - t_overlap / t_serial, 4),
        "hidden_compute_frac": round((t_serial - t_overlap) / t_comp, 4) if t_comp > 0 else None,
    }), flush=True)


def placement_replay(n_prefill, n_decode, fractions, n_layers):
    """Decode miss rates of the device cache's global LRU (every miss filled, and the q* split
    at the B_P / B_H measured on this host) against a prefill-time placement and a routing-blind
    placement, at equal capacity, replayed through ft_route_only / ft_cache_plan over synthetic
    routing traces with short-range locality (one trace per layer, n_layers layers)."""
    import torch
    import workloads
    from paper_2608_16157_amd import replay as rp
    bw = {"qwen3_decode": (53.92, 82.74), "dsv3_decode": (55.5, 44.9)}
    rows = []
    t0 = time.perf_counter()
    for name in ("qwen3_decode", "dsv3_decode"):
        c = workloads.CONFIGS[name]
        desc = dict(hidden=c.hidden, inter=c.inter, n_experts=c.n_experts, top_k=c.top_k,
                    gating=c.gating, w_dtype=c.w_dtype, x_dtype=c.x_dtype, n_slots=0, shared_slot=-1)
        traces = [workloads.routing_trace(name, n_prefill, n_decode, layer=l, device="cuda")
                  for l in range(n_layers)]
        for f in fractions:
            C = max(c.top_k, int(f * c.n_experts))
            rates = {}
            for pol in rp.POLICIES:
                miss = 0
                for tr in traces:
                    r = rp.replay(desc, tr, n_prefill, C, pol, *bw[name], k_max=c.top_k)
                    miss += int(r["misses"].sum())
                rates[pol] = round(miss / (n_layers * n_decode * c.top_k), 4)
            rows.append({"workload": name, "capacity": C, "capacity_frac": round(C / c.n_experts, 3),
                         "miss_rate": rates})
            print(json.dumps(rows[-1]), file=sys.stderr, flush=True)
    print(json.dumps({
        "measurement": "decode expert-read miss rate by placement policy (routing-trace replay)",
        "workload": f"synthetic routing traces: {n_prefill} prefill + {n_decode} decode tokens per "
                    f"layer, {n_layers} layers, topic segments of mean 64 tokens over 8 Zipf "
                    f"popularity rankings; B_P/B_H for 'split' as measured on this host",
        "policies": {"lru": "global LRU, every miss filled", "split": "global LRU with the q* split",
                     "prefill": "fixed top-C of the prefill routing", "blind": "fixed experts 0..C-1"},
        "results": rows, "seconds": round(time.perf_counter() - t0, 1)}), flush=True)


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(lay, tokens):
    """The float64 oracle on this host, on a bounded sample of the timed workload: one
    oracle.moe_partial call over ``tokens`` of one layer instance (every hit pair of those tokens
    plus the shared expert's rows; each touched expert's weights decoded once, as the oracle
    does), timed once on one thread and once on every CPU of this process's affinity mask."""
    import oracle
    import threadpoolctl
    from tests._util import oracle_inputs
    inp = oracle_inputs(lay)             # host copy, outside the timed part
    n_aff = len(os.sched_getaffinity(0))

    def run(threads):
        with threadpoolctl.threadpool_limits(limits=threads):
            t0 = time.perf_counter()
            oracle.moe_partial(*inp, tokens=tokens)
            return time.perf_counter() - t0

    t_all = run(n_aff)
    t_one = run(1)
    n = len(tokens)
    return {"value": round(n / t_all, 3), "unit": "tokens/s", "cores": n_aff, "kind": "oracle",
            "single_thread": {"value": round(n / t_one, 3), "unit": "tokens/s", "cores": 1,
                              "seconds": round(t_one, 2)},
            "affinity_cpus": n_aff, "cpu_model": _cpu_model(),
            "sample": f"one float64 oracle call over {n} tokens of layer instance 0 ({tokens[0]}, "
                      f"{tokens[1]}, ... {tokens[-1]}): all their hit pairs and shared-expert rows, "
                      f"each touched expert decoded once; {t_all:.1f} s on {n_aff} threads (BLAS "
                      f"pool limited to the affinity mask; the decodes are single-threaded numpy), "
                      f"{t_one:.1f} s on one thread"}


def measure_forward(config, T, n_layers, steps, warmup, hip, combine=0, act_quant=0, layers=None):
    """Time ``steps`` back-to-back ft_moe_forward calls over ``n_layers`` rotating instances of
    ``config`` at T tokens (inputs resident in HBM), then the same steps with stage events.
    Returns the throughput, the per-stage times and the dominant kernel's roofline, and the
    layer instances (for the CPU baseline).  act_quant selects the optional fp8-activation mode;
    ``layers`` reuses instances built by an earlier call."""
    import torch
    import paper_2608_16157_amd as ftm
    import workloads
    cfg = workloads.CONFIGS[config]
    if layers is None:
        print(f"# building {n_layers} layer instances of {config} T={T}", file=sys.stderr, flush=True)
        layers = [workloads.make_layer(config, T, layer=i, device="cuda") for i in range(n_layers)]
    desc = dict(layers[0].desc(), combine=combine, act_quant=act_quant)
    ws = ftm.alloc_workspace(desc, T)
    routes = [ftm.RouteBuffers(T, cfg.top_k, cfg.n_experts) for _ in layers]
    out = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
    banks = [ftm.banks_of(l) for l in layers]

    def step(i, events=None):
        j = i % len(layers)
        l = layers[j]
        if events is None:
            ftm.ft_moe_forward(desc, banks[j], l.logits, l.slot_table, l.x, T, out, routes[j], ws)
        else:
            ftm.ft_moe_forward_profiled(desc, banks[j], l.logits, l.slot_table, l.x, T, out,
                                        routes[j], ws, events)

    for i in range(len(layers)):          # route every instance once (setup, untimed)
        step(i)
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    work = [algorithmic_work(l, r, act_quant) for l, r in zip(layers, routes)]
    K = steps
    stream = torch.cuda.current_stream().cuda_stream
    start, stop = hip.create(), hip.create()

    # timed region 1: plain back-to-back steps -> throughput
    torch.cuda.synchronize()
    hip.hip.hipEventRecord(start, stream)
    for i in range(K):
        step(i)
    hip.hip.hipEventRecord(stop, stream)
    torch.cuda.synchronize()
    total_ms = hip.elapsed_ms(start, stop)
    ms_step = total_ms / K

    # timed region 2: the same steps with HIP events at the stage boundaries, recorded by the
    # library on its stream -> per-kernel durations (the events add gaps between kernels, so
    # this region is not used for throughput).  Timing-only events without the system-scope
    # fence, whose cache writeback would otherwise be charged to the stage after each boundary.
    stage_ev = [[hip.create(HIP_EVENT_DISABLE_SYSTEM_FENCE) for _ in range(ftm.FT_PROF_STAGES + 1)]
                for _ in range(K)]
    torch.cuda.synchronize()
    for i in range(K):
        step(i, stage_ev[i])
    torch.cuda.synchronize()
    stage_ms = [[hip.elapsed_ms(e[s], e[s + 1]) for s in range(ftm.FT_PROF_STAGES)] for e in stage_ev]
    for e in stage_ev:
        for ev in e:
            hip.destroy(ev)
    hip.destroy(start)
    hip.destroy(stop)

    step_work = [work[i % len(layers)] for i in range(K)]
    layer_bytes = sum(w["layer_bytes"] for w in step_work) / K
    layer_flops = sum(w["flops"] for w in step_work) / K
    gu_ms = sum(s[1] for s in stage_ms) / K
    gu_bytes = sum(w["gateup_bytes"] for w in step_work) / K
    gu_flops = sum(w["gateup_flops"] for w in step_work) / K
    stage_avg = [sum(s[j] for s in stage_ms) / K for j in range(ftm.FT_PROF_STAGES)]
    mfma_path = T >= 256      # the library's many-token (MFMA GEMM) path
    traffic = measured_traffic(f"{config}:T{T}" + (":fp8act" if act_quant else ""))
    if mfma_path and act_quant:
        # fp8 activations: fp8 x fp8 products on the matrix cores, against the fp8 dense peak
        achieved = gu_flops / (gu_ms / 1e3) / 1e12
        roof = {"kernel": "grouped gate/up GEMM, fp8 x fp8 + SiLU-mul (grouped_gemm<fp8 activations, gate/up>)",
                "bound": "mfma", "achieved": round(achieved, 1), "peak": MFMA_PEAK_TFLOPS["fp8"],
                "unit": "TFLOP/s", "frac": round(achieved / MFMA_PEAK_TFLOPS["fp8"], 4),
                "traffic": traffic, "flops_per_launch": round(gu_flops),
                "bytes_per_launch": round(gu_bytes), "ms_per_launch": round(gu_ms, 5)}
    elif mfma_path:
        # fp8 and MXFP4 weights are widened to bf16 in registers, so every contraction runs on
        # bf16 MFMA
        achieved = gu_flops / (gu_ms / 1e3) / 1e12
        roof = {"kernel": "grouped gate/up GEMM + SiLU-mul (grouped_gemm<gate/up>)", "bound": "mfma",
                "achieved": round(achieved, 1), "peak": MFMA_PEAK_TFLOPS["bf16"], "unit": "TFLOP/s",
                "frac": round(achieved / MFMA_PEAK_TFLOPS["bf16"], 4),
                "traffic": traffic, "flops_per_launch": round(gu_flops),
                "bytes_per_launch": round(gu_bytes), "ms_per_launch": round(gu_ms, 5)}
    else:
        achieved = gu_bytes / (gu_ms / 1e3) / 1e9
        roof = {"kernel": "grouped gate/up GEMV + SiLU-mul (grouped_gemv<gate/up>)", "bound": "hbm",
                "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "bytes_per_launch": round(gu_bytes), "ms_per_launch": round(gu_ms, 5)}
    wdt = {0: "f32", 1: "bf16", 2: "fp8 e4m3 + 128x128 float32 block scales, widened exactly to bf16",
           3: "MXFP4, widened exactly to bf16"}[cfg.w_dtype]
    if act_quant:
        wdt = ("fp8 e4m3 + 128x128 float32 block scales, activations quantised to fp8 e4m3 per token "
               "and 128 channels with power-of-two scales (optional mode, not the exact method)")
    res = {
        "value": round(T * K / (total_ms / 1e3), 1),
        "ms_per_step": round(ms_step, 5),
        "workload": f"{config}: MoE layer over a GPU expert cache, T={T} tokens, E={cfg.n_experts} "
                    f"top-{cfg.top_k}, H={cfg.hidden} I={cfg.inter}, weights {wdt}, "
                    f"{layers[0].n_slots} slots, {n_layers} rotating layer instances",
        "layer_hbm_gbps": round(layer_bytes / (ms_step / 1e3) / 1e9, 1),
        "layer_hbm_frac": round(layer_bytes / (ms_step / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
        "layer_tflops": round(layer_flops / (ms_step / 1e3) / 1e12, 2),
        "layer_mfma_frac": round(layer_flops / (ms_step / 1e3) / 1e12 /
                                 MFMA_PEAK_TFLOPS["fp8" if act_quant and mfma_path else "bf16"], 4),
        "stage_ms": {"route": round(stage_avg[0], 5), "gate_up": round(stage_avg[1], 5),
                     "down": round(stage_avg[2], 5), "combine": round(stage_avg[3], 5)},
        "roofline": roof,
    }
    return res, layers


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="dsv3_prefill")
    ap.add_argument("--tokens", type=int, default=8192)
    ap.add_argument("--layers", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--decode-extras", default="qwen3_decode:32,dsv3_decode:64",
                    help="decode points (config:T, comma-separated) timed after the headline in the "
                         "same run, reported under 'decode'; '' for none")
    ap.add_argument("--act-quant", type=int, default=0,
                    help="1: the optional fp8-activation mode (FT_ACT_FP8_1x128_POW2) for --config")
    ap.add_argument("--fp8-act-extra", type=int, default=1,
                    help="with an fp8 many-token headline, also time the fp8-activation mode on the same "
                         "instances, reported under 'fp8_act' (0: skip)")
    ap.add_argument("--measure-bandwidths", action="store_true",
                    help="measure B_P (fills over PCIe) and B_H (CPU branch) for --config, then exit")
    ap.add_argument("--hybrid", action="store_true",
                    help="time complete decode steps with fills and the CPU branch, then exit")
    ap.add_argument("--cache-plan", action="store_true",
                    help="time device-side cache control (ft_route_only + ft_cache_plan) per decode step")
    ap.add_argument("--slots", type=int, default=64, help="cache slots for --hybrid / --cache-plan")
    ap.add_argument("--b-pcie", type=float, default=50.0, help="B_P (GB/s) for --hybrid")
    ap.add_argument("--b-host", type=float, default=60.0, help="B_H (GB/s) for --hybrid")
    ap.add_argument("--max-fill", type=int, default=8, help="K for --hybrid")
    ap.add_argument("--prefill-pipeline", action="store_true",
                    help="time full-layer double-buffered prefill over --layers layers (overlapped "
                         "and serialised), then exit")
    ap.add_argument("--replay", action="store_true",
                    help="replay synthetic decode routing traces under each placement policy "
                         "(--layers traces per workload), then exit")
    ap.add_argument("--calibrate-copy", type=int, metavar="MIB",
                    help="run only a plain copy kernel of MIB MiB (counter calibration)")
    ap.add_argument("--ingest-traffic", nargs="+",
                    metavar="KEY KERNEL FETCH_CSV WRITE_CSV CAL_FETCH_CSV CAL_WRITE_CSV CAL_BYTES [PER_KERNEL]",
                    help="record per-launch HBM traffic from rocprofv3 counter CSVs and exit "
                         "(PER_KERNEL: a kernel dispatched once per layer forward, for a stage "
                         "issued as several dispatches)")
    args = ap.parse_args()
    if args.ingest_traffic:
        a = args.ingest_traffic
        if len(a) not in (7, 8):
            ap.error("--ingest-traffic takes 7 or 8 arguments")
        ingest_traffic(a[0], a[1], a[2], a[3], a[4], a[5], int(a[6]), a[7] if len(a) == 8 else None)
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one MI355X: this library runs the MoE layer over a GPU expert cache "
              "on a single GPU (no sharding or collectives); run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2608_16157_amd as ftm
    import workloads

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return
    if args.measure_bandwidths:
        measure_bandwidths(args.config, 8, 10)
        return
    if args.replay:
        placement_replay(1024, 2048, (0.11, 0.25, 0.37, 0.5, 0.75), min(args.layers, 4))
        return
    if args.prefill_pipeline:
        prefill_pipeline(args.config, args.tokens, args.layers, max(1, args.steps))
        return
    if args.cache_plan:
        cache_plan_timing(args.config, args.tokens, args.steps, args.warmup, args.slots, args.b_pcie,
                          args.b_host, args.max_fill)
        return
    if args.hybrid:
        hybrid_decode(args.config, args.tokens, args.steps, args.warmup, args.slots, args.b_pcie,
                      args.b_host, args.max_fill)
        return
    ftm.load()
    hip = HipEvents()
    T = args.tokens
    res, layers = measure_forward(args.config, T, args.layers, args.steps, args.warmup, hip,
                                  act_quant=args.act_quant)
    cfg = workloads.CONFIGS[args.config]
    line = {
        "metric": METRIC,
        "value": res["value"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.w_dtype != 0 else "f32",
        "data": "synthetic",
        "config": {"workload": res["workload"], "tokens": T, "layers": args.layers},
    }
    for k in ("layer_hbm_gbps", "layer_hbm_frac", "layer_tflops", "layer_mfma_frac", "stage_ms",
              "roofline"):
        line[k] = res[k]
    if not args.no_cpu_baseline:
        print("# timing the CPU oracle", file=sys.stderr, flush=True)
        if T <= 64:
            toks = list(range(T))
        else:   # eight tokens from each eighth of the chunk (every hot-set segment of dsv3_prefill)
            toks = sorted({i * (T // 8) + j for i in range(8) for j in range(min(8, T // 8))})
        line["cpu_baseline"] = cpu_baseline(layers[0], toks)
    if args.fp8_act_extra and not args.act_quant and cfg.w_dtype == workloads.DT_FP8 and T >= 256:
        # the optional fp8-activation mode on the same layer instances (not the headline: the
        # exact mode is the paper's method)
        ra, _ = measure_forward(args.config, T, args.layers, args.steps, args.warmup, hip,
                                act_quant=ftm.FT_ACT_FP8_1x128_POW2, layers=layers)
        line["fp8_act"] = {k: ra[k] for k in ("value", "ms_per_step", "workload", "layer_tflops",
                                               "layer_mfma_frac", "stage_ms", "roofline")}
        line["fp8_act"]["unit"] = "tokens/s"
    del layers
    torch.cuda.empty_cache()
    # decode points of the metric's other half (achieved HBM bandwidth), timed in the same run
    if args.decode_extras:
        extras = {}
        for spec in args.decode_extras.split(","):
            name, t = spec.split(":")
            n_dec = 16 if name.startswith("qwen3") else 8
            r, lays = measure_forward(name, int(t), n_dec, max(10 * args.steps, 100), args.warmup, hip)
            del lays
            torch.cuda.empty_cache()
            ra, lays = measure_forward(name, int(t), n_dec, max(10 * args.steps, 100), args.warmup, hip,
                                       combine=ftm.FT_COMBINE_ATOMIC)
            del lays
            torch.cuda.empty_cache()
            e = {k: r[k] for k in ("value", "ms_per_step", "workload", "layer_hbm_gbps", "layer_hbm_frac",
                                   "stage_ms", "roofline")}
            e.update(unit="tokens/s", steps=max(10 * args.steps, 100), combine="ordered (bit-reproducible)",
                     atomic_combine={k: ra[k] for k in ("value", "ms_per_step", "layer_hbm_gbps",
                                                        "layer_hbm_frac", "stage_ms")})
            extras[f"{name}:T{t}"] = e
        line["decode"] = extras
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
