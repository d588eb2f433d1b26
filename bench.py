"""Benchmark of the calibration-replay hot path on one MI355X.

A step is one kvr_bootstrap call on the two-tier workload: 4,096 bootstrap
resamples of 65,536 waits x 64 GPU-tier timers x 257 host timers (256 plus
host-retain) x 32 loads = 1.413e14 (sample, policy, load) cost evaluations,
with the per-resample selection fused.  Inputs are resident in HBM before
the timed region.  Prints one JSON line.

The roofline of the dominant kernel (the brute-force grid) is the fp64
vector ALU: one FMA (2 flops) per evaluation is the algorithmic work; the
peak is MI355X's 78.6 TFLOP/s fp64 vector rate (256 CUs x 4 SIMDs x 16 lanes
x 2 flops x 2.4 GHz).  The cpu_baseline leg times the CPU oracle, as it
stands, on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

FP64_PEAK_TFLOPS = 78.6
HBM_PEAK_GBS = 8000.0


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="twotier-4096x64k")
    ap.add_argument("--resamples", type=int, default=None,
                    help="truncate the bootstrap batch (for quick local runs)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=1,
                    help="bootstrap rows the CPU oracle evaluates for cpu_baseline")
    ap.add_argument("--paths", action="store_true",
                    help="also time the other paths (sorted closed form, plain grid)")
    ap.add_argument("--traffic-json", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="HBM bytes per launch of the grid kernel from rocprofv3 counters")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1 "
                                   "(the bootstrap batch would shard by resample with no "
                                   "exchange, see DESIGN.md)"}))
        return 2

    import numpy as np
    import torch

    import paper_2608_30830_amd as kvr
    import workloads

    log(f"[bench] workload {args.workload}: generating inputs")
    wl = workloads.make(args.workload, resamples=args.resamples)
    pf = wl.platform
    prices = kvr.kvr_prices_from_platform(wl.kv_bytes_per_token, pf["hbm_usable_bytes"],
                                          pf["host_link_bytes_per_s"],
                                          pf["prefill_tokens_per_s"], pf["n_gpu"],
                                          pf["host_slots_c2"], pf["w_ref_s"])
    grid = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    w = torch.as_tensor(wl.wait_s, dtype=torch.float64).to(dev)
    T = torch.as_tensor(wl.ctx_tokens, dtype=torch.int32).to(dev)
    idx = torch.as_tensor(wl.idx, dtype=torch.int32).to(dev)
    call = kvr.BootstrapCall(w, T, idx, prices, grid)
    evals = wl.evaluations
    stream = torch.cuda.current_stream()

    log(f"[bench] warmup {args.warmup} step(s)")
    for _ in range(args.warmup):
        call.launch()
    torch.cuda.synchronize()
    st = call.status()
    if st != kvr.KVR_OK:
        raise kvr.KvrError(st, "warmup")

    log(f"[bench] timing {args.steps} step(s)")
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    stops = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        starts[i].record(stream)
        call.launch()
        stops[i].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ev_ms = [a.elapsed_time(b) for a, b in zip(starts, stops)]
    ms_per_step = 1000.0 * wall / args.steps
    launch_ms = sum(ev_ms) / len(ev_ms)
    log(f"[bench] {ms_per_step:.1f} ms/step wall, {launch_ms:.1f} ms/launch (events)")

    achieved = 2.0 * evals / (launch_ms * 1e-3) / 1e12
    traffic = None
    if os.path.exists(args.traffic_json):
        with open(args.traffic_json) as fh:
            tj = json.load(fh)
        if tj.get("workload") == args.workload and tj.get("resamples") == wl.n_resamples:
            traffic = tj.get("bytes_per_launch")
    out = {
        "metric": "sample×policy cost evaluations/sec at 1 GPU; % of HBM/FP64 roofline",
        "value": evals / (ms_per_step * 1e-3),
        "unit": "evaluations/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": args.workload, "samples": wl.n, "resamples": wl.n_resamples,
                   "resample_len": wl.m, "t1_timers": int(wl.t1.size),
                   "t2_timers": int(wl.t2.size), "loads": int(wl.lam.size),
                   "evaluations_per_step": evals, "method": "brute-force grid, fused selection"},
        "roofline": {"bound": "alu", "achieved": achieved, "peak": FP64_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / FP64_PEAK_TFLOPS,
                     "traffic": traffic, "kernel": "grid_kernel<32,true>",
                     "launch_ms": launch_ms,
                     "note": "2 flops (one fp64 FMA) per evaluation; launch_ms spans the whole "
                             "call (grid kernel plus four small kernels)"},
    }

    if args.paths:
        out["paths"] = time_paths(kvr, workloads, torch)

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_rows)

    print(json.dumps(out), flush=True)
    return 0


def time_paths(kvr, workloads, torch):
    """Milliseconds per call of the other entry points on their workloads."""
    res = {}
    for name, method in (("weibull-1m", kvr.KVR_BRUTE), ("weibull-1m", kvr.KVR_SORTED),
                         ("mix-64k", kvr.KVR_BRUTE), ("mix-64k", kvr.KVR_SORTED)):
        wl = workloads.make(name)
        pf = wl.platform
        pr = kvr.kvr_prices_from_platform(wl.kv_bytes_per_token, pf["hbm_usable_bytes"],
                                          pf["host_link_bytes_per_s"],
                                          pf["prefill_tokens_per_s"])
        g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
        w = torch.as_tensor(wl.wait_s).cuda()
        T = torch.as_tensor(wl.ctx_tokens).cuda()
        out = torch.empty((wl.lam.size, wl.t1.size, wl.t2.size), dtype=torch.float64, device="cuda")
        kvr.kvr_cost_grid(w, T, pr, g, method=method, out=out)
        ws = None
        times = []
        for _ in range(5):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            kvr.kvr_cost_grid(w, T, pr, g, method=method, out=out, workspace=ws, check=False)
            b.record()
            torch.cuda.synchronize()
            times.append(a.elapsed_time(b))
        ms = sorted(times)[len(times) // 2]
        key = f"{name}/{'sorted' if method == kvr.KVR_SORTED else 'brute'}"
        res[key] = {"ms": ms, "evaluations_per_s": wl.evaluations / (ms * 1e-3)}
        log(f"[bench] path {key}: {ms:.3f} ms")
    return res


def cpu_baseline(wl, rows: int):
    """The oracle double loop on the first ``rows`` bootstrap rows, all policies
    and loads; scaled to evaluations per second."""
    import oracle
    pr = oracle.workload_prices(wl)
    log(f"[bench] cpu baseline: oracle on {rows} row(s) with {oracle.num_threads()} threads")
    t0 = time.perf_counter()
    for r in range(rows):
        oracle.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam, idx_row=wl.idx[r])
    dt = time.perf_counter() - t0
    ev = rows * wl.m * wl.t1.size * wl.t2.size * wl.lam.size
    return {"value": ev / dt, "unit": "evaluations/s", "cores": oracle.num_threads(),
            "kind": "oracle", "seconds": dt,
            "sample": f"{rows} of {wl.n_resamples} bootstrap rows, every policy and load "
                      f"({ev:.3e} evaluations)"}


if __name__ == "__main__":
    sys.exit(main())
