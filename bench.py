#!/usr/bin/env python3
"""Benchmark of the MoE layer over a GPU expert cache on one MI355X.

One step = one ft_moe_forward call (routing, hit/miss split, permutation, grouped SwiGLU expert
FFN over the cache-resident experts, gate-weighted combine) on one synthetic layer instance with
its inputs already resident in HBM.  Steps rotate over --layers distinct layer instances, each
with its own slot-pool weights and routing, so a cycle's working set exceeds the 256 MB
Infinity Cache and weights really stream from HBM.

Prints ONE JSON line: tokens/s (whole job), ms per step, the dominant kernel's roofline
fraction (algorithmic bytes of one launch / its HIP-event-timed duration on the library's
stream), and the CPU oracle timed on a bounded sample on this host.
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
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "fp8": 5000.0}


class HipEvents:
    """hipEvent_t handles through the HIP runtime torch already loaded."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so.7")
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self):
        ev = ctypes.c_void_p()
        if self.hip.hipEventCreate(ctypes.byref(ev)) != 0:
            raise RuntimeError("hipEventCreate failed")
        return ev.value

    def elapsed_ms(self, a, b) -> float:
        ms = ctypes.c_float()
        if self.hip.hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(a), ctypes.c_void_p(b)) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def destroy(self, ev):
        self.hip.hipEventDestroy(ctypes.c_void_p(ev))


def expert_bytes(lay):
    """Bytes of one complete expert (W1, W3, W2 and block scales) and of its W13 part."""
    H, I = lay.hidden, lay.inter
    wb = {0: 4, 1: 2, 2: 1}[lay.w_dtype]
    s13 = (2 * I // 128) * (H // 128) * 4 if lay.w_dtype == 2 else 0
    s2 = (H // 128) * (I // 128) * 4 if lay.w_dtype == 2 else 0
    w13 = 2 * I * H * wb + s13
    return w13 + H * I * wb + s2, w13


def algorithmic_work(lay, route):
    """Bytes the layer must move and flops it must do, from the realised routing."""
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
    flops = rows * 6 * H * I
    return dict(layer_bytes=layer_bytes, gateup_bytes=gateup_bytes, flops=flops, u_hit=u_hit,
                n_hit=n_hit, rows=rows)


def cpu_baseline(layers, budget_s):
    """The float64 oracle on this host over a bounded sample of the same layer instances."""
    import oracle
    from tests._util import oracle_inputs
    try:
        import threadpoolctl
        info = threadpoolctl.threadpool_info()
        cores = max([i.get("num_threads", 1) for i in info] or [1])
    except Exception:
        cores = 1
    done_tokens, elapsed, used = 0, 0.0, 0
    for lay in layers:
        inp = oracle_inputs(lay)          # host copy, outside the timed part
        t0 = time.perf_counter()
        oracle.moe_partial(*inp)
        elapsed += time.perf_counter() - t0
        done_tokens += lay.tokens
        used += 1
        if elapsed >= budget_s:
            break
    return {"value": done_tokens / elapsed, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"{used} of the {len(layers)} layer instances ({done_tokens} tokens), "
                      f"{elapsed:.1f} s of float64 oracle time"}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="qwen3_decode")
    ap.add_argument("--tokens", type=int, default=32)
    ap.add_argument("--layers", type=int, default=16)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one MI355X: the MoE layer over a GPU expert cache runs on a single "
              "GPU (no sharding or collectives in this build); run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2608_16157_amd as ftm
    import workloads

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    ftm.load()
    cfg = workloads.CONFIGS[args.config]
    T = args.tokens
    print(f"# building {args.layers} layer instances of {args.config} T={T}", file=sys.stderr, flush=True)
    layers = [workloads.make_layer(args.config, T, layer=i, device="cuda") for i in range(args.layers)]
    desc = layers[0].desc()
    ws = ftm.alloc_workspace(desc, T)
    routes = [ftm.RouteBuffers(T, cfg.top_k, cfg.n_experts) for _ in layers]
    out = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
    banks = [ftm.banks_of(l) for l in layers]

    def step(i, events=None):
        l = layers[i % len(layers)]
        if events is None:
            ftm.ft_moe_forward(desc, banks[i % len(layers)], l.logits, l.slot_table, l.x, T, out,
                               routes[i % len(layers)], ws)
        else:
            ftm.ft_moe_forward_profiled(desc, banks[i % len(layers)], l.logits, l.slot_table, l.x, T,
                                        out, routes[i % len(layers)], ws, events)

    for i in range(len(layers)):          # route every instance once (setup, untimed)
        step(i)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    work = [algorithmic_work(l, r) for l, r in zip(layers, routes)]

    hip = HipEvents()
    K = args.steps
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
    # this region is not used for throughput)
    stage_ev = [[hip.create() for _ in range(ftm.FT_PROF_STAGES + 1)] for _ in range(K)]
    torch.cuda.synchronize()
    for i in range(K):
        step(i, stage_ev[i])
    torch.cuda.synchronize()
    stage_ms = [[hip.elapsed_ms(e[s], e[s + 1]) for s in range(ftm.FT_PROF_STAGES)] for e in stage_ev]
    for e in stage_ev:
        for ev in e:
            hip.destroy(ev)

    tokens_per_s = T * K / (total_ms / 1e3)
    step_work = [work[i % len(layers)] for i in range(K)]
    layer_bytes = sum(w["layer_bytes"] for w in step_work) / K
    layer_flops = sum(w["flops"] for w in step_work) / K
    gu_ms = sum(s[1] for s in stage_ms) / K
    gu_bytes = sum(w["gateup_bytes"] for w in step_work) / K
    stage_avg = [sum(s[j] for s in stage_ms) / K for j in range(ftm.FT_PROF_STAGES)]

    achieved = gu_bytes / (gu_ms / 1e3) / 1e9
    dtype = {0: "f32", 1: "bf16", 2: "fp8e4m3->bf16"}[cfg.w_dtype]
    res = {
        "metric": METRIC,
        "value": round(tokens_per_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.w_dtype != 0 else "f32",
        "data": "synthetic",
        "config": {
            "workload": f"{args.config}: MoE layer over a GPU expert cache, T={T} tokens, "
                        f"E={cfg.n_experts} top-{cfg.top_k}, H={cfg.hidden} I={cfg.inter}, "
                        f"weights {dtype}, {layers[0].n_slots} slots, "
                        f"{args.layers} rotating layer instances",
            "tokens": T, "layers": args.layers,
        },
        "layer_hbm_gbps": round(layer_bytes / (ms_step / 1e3) / 1e9, 1),
        "layer_hbm_frac": round(layer_bytes / (ms_step / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
        "layer_tflops": round(layer_flops / (ms_step / 1e3) / 1e12, 2),
        "stage_ms": {"route": round(stage_avg[0], 5), "gate_up": round(stage_avg[1], 5),
                     "down": round(stage_avg[2], 5), "combine": round(stage_avg[3], 5)},
        "roofline": {
            "kernel": "grouped gate/up projection + SiLU-mul",
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": None,
            "bytes_per_launch": round(gu_bytes),
            "ms_per_launch": round(gu_ms, 5),
        },
    }
    if not args.no_cpu_baseline:
        print("# timing the CPU oracle", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(layers, args.cpu_seconds)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
