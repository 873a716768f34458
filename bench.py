#!/usr/bin/env python3
"""Benchmark of the expert-slot-cache MoE layer on one MI355X.

Workload (default): the A3B-shaped Q8_0 decode stack -- 48 MoE layers, hidden
2048, 128 experts, top-8, expert intermediate 768, weights N(0, 0.02)
quantised to Q8_0, fp32 router N(0, 0.05), 96 tokens decoded one at a time
with AR(1) hidden states (rho 0.8), 19 slots per layer (15%), LRU, the whole
28.7 GiB expert store in pinned host memory.  Data are synthetic and seeded.

One step = one full 96-token x 48-layer decode from a cold cache (every
layer's slot table reset), the layers chained h <- h + moe(rmsnorm(h)) on the
GPU (the library's residual and pre-norm flags).
value = decoded tokens / wall seconds over the timed steps, inputs already in
HBM / pinned memory when timing starts.

Printed: one JSON line with the contract fields plus
  roofline      the gate/up dequant-GEMV kernel (the largest share of expert
                bytes) against the 8 TB/s HBM peak, from HIP events around
                every launch in the timed region;
  cpu_baseline  the CPU oracle on a bounded sample of the same workload;
  extra         hit rate, materialised bytes/token, copy GB/s vs the measured
                host-to-device peak, per-kernel timings.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# PCIe 5.0 x16, one direction: 32 GT/s x 16 lanes x 128/130 encoding / 8 bits
PCIE_PEAK_GBS = 32.0 * 16 * 128 / 130 / 8
BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
HBM_BYTES = 288 * 10**9    # MI355X HBM3E capacity


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="a3b_decode",
                    choices=["a3b_decode", "q4_decode", "tiny", "a3b_prefill"])
    ap.add_argument("--budget", type=int, default=None, help="slots per layer (default: workload's)")
    ap.add_argument("--rho", type=float, default=None)
    ap.add_argument("--no-timing", action="store_true", help="no HIP events around kernels")
    ap.add_argument("--timing-stride", type=int, default=16,
                    help="bracket one layer call in this many with HIP events")
    ap.add_argument("--copy-mode", default="kernel", choices=["kernel", "split", "side", "sdma"],
                    help="kernel: miss copies fused with gate/up in one launch (default); "
                         "split: copy kernel then gate/up kernel; side: hipMemcpyAsync on a "
                         "side stream overlapped with the hit experts; sdma: hipMemcpyAsync "
                         "on the compute stream")
    ap.add_argument("--cpu-sample-tokens", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "gateup_a3b_q8_traffic.json"),
                    help="JSON with the measured HBM bytes per gate/up launch (rocprofv3 --pmc); used "
                         "only if it was taken on the current kernels.hip and this workload")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="after the run, copy 256 MiB device-to-device 4 times with torch (a plain "
                         "copy kernel of known size, to scale the FETCH_SIZE / WRITE_SIZE counters)")
    return ap.parse_args()


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the expert-slot-cache path has no multi-GPU "
              "mode in this build (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    from paper_2607_09686_amd import (KIND_COPY, KIND_DOWN, KIND_GATEUP, KIND_ROUTER, HostBuffer,
                                      MoeCache, plan_percent, probe_h2d)

    wl = synth.WORKLOADS[args.workload]
    # slots per layer from the workload's cache percentage, by the library's static planner;
    # the plan's lower bound (router weights + expert slots, no KV cache on this path) is
    # checked against the GPU's HBM
    model = {"n_layers": wl.n_layers, "n_experts": wl.n_experts, "top_k": wl.top_k,
             "payload_bytes": wl.payload_bytes, "common_bytes": wl.n_layers * wl.hidden * wl.n_experts * 4,
             "kv_bytes_per_token": 0, "overhead_bytes": 0, "target_bytes": HBM_BYTES}
    plan = plan_percent(model, wl.cache_percent)
    if plan["slots_per_layer"] != wl.budget_slots:
        raise RuntimeError(f"planner gives {plan['slots_per_layer']} slots, workload {wl.budget_slots}")
    budget = args.budget or wl.budget_slots
    rho = wl.rho if args.rho is None else args.rho
    torch.cuda.set_device(0)

    log(f"workload {wl.name}: L={wl.n_layers} H={wl.hidden} E={wl.n_experts} k={wl.top_k} "
        f"I={wl.inter} {wl.qtype} C={budget} T={wl.n_tokens} rho={rho}")
    t0 = time.time()
    hb = HostBuffer(wl.store_bytes)
    log(f"pinned {wl.store_bytes / 2**30:.2f} GiB in {time.time() - t0:.1f} s")
    t0 = time.time()
    synth.expert_store(wl, out=hb.array)
    log(f"generated expert store in {time.time() - t0:.1f} s")
    R = synth.router(wl)
    X = synth.hidden(wl, rho=rho)
    Rd = torch.from_numpy(R).cuda()
    Xd = torch.from_numpy(X).cuda()

    # measured pinned host-to-device bandwidth: 64 expert-sized copies, one stream
    # (the probe reads n_chunks * chunk bytes of the store: keep it inside the buffer)
    n_small = min(64, wl.store_bytes // wl.payload_bytes)
    h2d_peak = probe_h2d(hb.ptr, wl.payload_bytes, n_small, 1)
    h2d_big = probe_h2d(hb.ptr, 1 << 30, 4, 1) if wl.store_bytes >= 4 << 30 else None
    log(f"H2D probe: {h2d_peak:.1f} GB/s ({n_small} expert-size copies), {h2d_big} GB/s (1 GiB copies)")

    timing = not args.no_timing
    cache = MoeCache(wl.n_layers, wl.n_experts, wl.top_k, wl.hidden, wl.inter, wl.qtype, hb.ptr,
                     wl.store_bytes, budget, stream=torch.cuda.current_stream(), residual=True,
                     prenorm=True, timing=timing, copy_mode=args.copy_mode)
    if timing:
        cache.set_timing_stride(args.timing_stride)
    h = torch.empty(wl.hidden, dtype=torch.float32, device="cuda")
    y = torch.empty_like(h)

    prefill = wl.mode == "prefill"
    if prefill:
        h = torch.empty_like(Xd)
        y = torch.empty_like(Xd)

    def step():
        nonlocal h, y
        cache.reset()
        if prefill:  # the whole chunk through every layer
            h.copy_(Xd)
            for l in range(wl.n_layers):
                cache.layer_forward(h, Rd[l], l, y, n_tokens=wl.n_tokens)
                h, y = y, h
            return
        for t in range(wl.n_tokens):
            h.copy_(Xd[t])
            for l in range(wl.n_layers):
                cache.layer_forward(h, Rd[l], l, y, n_tokens=1)
                h, y = y, h

    kinds = ((KIND_ROUTER, "router"), (KIND_GATEUP, "gateup"), (KIND_DOWN, "down"),
             (KIND_COPY, "copy"))
    for i in range(args.warmup):
        step()
        log(f"warmup step {i} done")
    torch.cuda.synchronize()
    counters = [0, 0, 0, 0]
    acc = {name: dict(launches=0, total_ms=0.0, bytes=0, flops=0) for _, name in kinds}
    ts = time.perf_counter()
    for i in range(args.steps):
        step()
        # one step's counters and event timings, read before the next step's reset
        counters = [a + b for a, b in zip(counters, cache.counters().as_tuple())]
        if timing:
            for kind, name in kinds:
                s = cache.kernel_stats(kind)
                a = acc[name]
                a["launches"] += s.launches
                a["total_ms"] += s.total_ms
                a["bytes"] += s.bytes
                a["flops"] += s.flops
    torch.cuda.synchronize()
    dt = time.perf_counter() - ts
    log(f"timed {args.steps} steps in {dt:.2f} s")
    tokens = args.steps * wl.n_tokens
    hits, misses, evictions, mbytes = counters
    stats = {}
    for _, name in kinds:
        a = acc[name]
        if a["launches"]:
            stats[name] = dict(a, avg_us=1e3 * a["total_ms"] / a["launches"],
                               gb_per_s=a["bytes"] / (a["total_ms"] * 1e6) if a["total_ms"] else None)
    result = {
        "metric": ("MoE-layer prefill tokens/s; expert-FFN MFMA utilisation; materialized bytes/token"
                   if prefill else
                   "MoE-layer decode tokens/s; expert-FFN HBM GB/s; materialized bytes/token"),
        "value": tokens / dt,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * dt / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if prefill else "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "n_layers": wl.n_layers, "hidden": wl.hidden,
                   "n_experts": wl.n_experts, "top_k": wl.top_k, "inter": wl.inter,
                   "qtype": wl.qtype, "budget_slots": budget, "n_tokens": wl.n_tokens, "rho": rho,
                   "copy_mode": args.copy_mode,
                   "global_batch": wl.n_tokens if prefill else 1, "seq_len": wl.n_tokens,
                   "parallelism": "none"},
    }
    if timing and prefill:
        gu = stats["gateup"]
        avg_s = gu["total_ms"] / 1e3 / max(1, gu["launches"])
        per_launch_flops = gu["flops"] / max(1, gu["launches"])
        achieved = per_launch_flops / avg_s / 1e12
        result["roofline"] = {"bound": "mfma", "kernel": "pf_gateup_kernel<8>", "achieved": achieved,
                              "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                              "frac": achieved / BF16_PEAK_TFLOPS, "traffic": None,
                              "flops_per_launch": per_launch_flops, "avg_launch_us": avg_s * 1e6}
        ffn_ms = stats["gateup"]["total_ms"] + stats["down"]["total_ms"]
        ffn_bytes = stats["gateup"]["bytes"] + stats["down"]["bytes"]
    elif timing and "gateup" not in stats:
        # one launch copies the misses and runs gate/up for all routed experts: it is
        # the dominant kernel and the host link bounds it
        cp, n_calls = stats["copy"], max(1, stats["router"]["launches"])
        avg_s = cp["total_ms"] / 1e3 / n_calls
        per_launch_bytes = cp["bytes"] / n_calls
        achieved = per_launch_bytes / avg_s / 1e9
        result["roofline"] = {"bound": "pcie", "kernel": "copy_gateup_kernel<8>" if wl.qtype == "q8_0"
                              else "copy_gateup_kernel<2>", "achieved": achieved,
                              "peak": PCIE_PEAK_GBS, "unit": "GB/s", "frac": achieved / PCIE_PEAK_GBS,
                              "traffic": None, "bytes_per_launch": per_launch_bytes,
                              "avg_launch_us": avg_s * 1e6}
        ffn_ms = stats["down"]["total_ms"]
        ffn_bytes = stats["down"]["bytes"]
    elif timing:
        gu = stats["gateup"]
        per_launch_bytes = gu["bytes"] / max(1, gu["launches"])
        avg_s = gu["total_ms"] / 1e3 / max(1, gu["launches"])
        achieved = per_launch_bytes / avg_s / 1e9
        traffic = None
        if args.traffic and os.path.exists(args.traffic):
            import hashlib
            t = json.load(open(args.traffic))
            src = os.path.join(ROOT, "paper_2607_09686_amd", "csrc", "kernels.hip")
            cur = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
            if t.get("kernels_hip_sha256_16") == cur and t.get("workload") == wl.name and \
                    budget == wl.budget_slots:
                traffic = t["traffic_bytes_per_launch"]
        result["roofline"] = {"bound": "hbm", "kernel": "gateup_kernel<8>" if wl.qtype == "q8_0"
                              else "gateup_kernel<2>", "achieved": achieved, "peak": HBM_PEAK_GBS,
                              "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                              "bytes_per_launch": per_launch_bytes, "avg_launch_us": avg_s * 1e6}
        ffn_ms = stats["gateup"]["total_ms"] + stats["down"]["total_ms"]
        ffn_bytes = stats["gateup"]["bytes"] + stats["down"]["bytes"]
    result["extra"] = {
        "hit_rate": hits / max(1, hits + misses),
        "misses_per_token_layer": misses / (tokens * wl.n_layers),
        "materialized_bytes_per_token": mbytes / tokens,
        "evictions_per_step": evictions / args.steps,
        "us_per_layer_call": 1e6 * dt / (tokens * wl.n_layers),
        "h2d_peak_gb_per_s": h2d_peak,
        "h2d_1gib_gb_per_s": h2d_big,
        "static_plan": dict(plan, cache_percent=wl.cache_percent, target="HBM 288 GB"),
    }
    if timing and "copy" in stats:
        cp = stats["copy"]
        if prefill:
            fl = stats["gateup"]["flops"] + stats["down"]["flops"]
            result["extra"]["expert_ffn_tflops"] = fl / (ffn_ms * 1e9)
            result["extra"]["expert_ffn_frac_of_bf16_peak"] = fl / (ffn_ms * 1e9) / BF16_PEAK_TFLOPS
        result["extra"].update({
            "expert_ffn_gb_per_s": ffn_bytes / (ffn_ms * 1e6),
            "expert_ffn_frac_of_hbm_peak": ffn_bytes / (ffn_ms * 1e6) / HBM_PEAK_GBS,
            "expert_ffn_kernels": "gate/up + down" if "gateup" in stats else
                                  "down (gate/up runs inside the copy launch)",
            "copy_gb_per_s": cp["gb_per_s"],
            "copy_frac_of_best_measured_h2d": (cp["gb_per_s"] or 0) / max(h2d_peak, h2d_big or 0),
            "kernels": stats,
        })
    cache.close()
    if args.calibrate_copy:
        a = torch.empty(256 << 20, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        a.fill_(1)
        for _ in range(4):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    if not args.no_cpu_baseline:
        from threadpoolctl import threadpool_info
        from oracle.layer import run_stack
        n = args.cpu_sample_tokens
        log(f"cpu baseline: oracle on the first {n} tokens through all {wl.n_layers} layers")
        tc = time.perf_counter()
        if prefill:  # a bounded sample: n tokens of the chunk as one multi-token call per layer
            run_stack(X[:n], R, hb.array, wl, budget, decode=False, bf16=True, prenorm=True)
        else:
            run_stack(X[:n], R, hb.array, wl, budget, prenorm=True)
        cdt = time.perf_counter() - tc
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
        result["cpu_baseline"] = {"value": n / cdt, "unit": "tokens/s", "cores": threads,
                                  "kind": "oracle",
                                  "sample": f"first {n} of {wl.n_tokens} tokens, all {wl.n_layers} "
                                            f"layers, same inputs, fp64 numpy ({cdt:.1f} s)"}
    hb.free()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
