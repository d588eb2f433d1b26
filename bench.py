"""Benchmark of the calibration-replay hot path on one MI355X.

A step is one kvr_bootstrap call on the two-tier workload: 4,096 bootstrap
resamples of 65,536 waits x 64 GPU-tier timers x 257 host timers (256 plus
host-retain) x 32 loads = 1.413e14 (sample, policy, load) cost evaluations,
with the per-resample selection fused.  Inputs are resident in HBM before
the timed region.  Prints one JSON line.

The roofline of the dominant kernel (the brute-force grid kernel) is the
fp64 vector ALU: one FMA (2 flops) per evaluation is the algorithmic work;
the peak is MI355X's 78.6 TFLOP/s fp64 vector rate (256 CUs x 4 SIMDs x 16
lanes x 2 flops x 2.4 GHz).  Its duration is taken with HIP events that the
library records on the launch stream right before and after that kernel.
The cpu_baseline leg times the CPU oracle, as it stands, on a bounded sample
of the same workload.

``--copy-calibration`` instead runs one plain device-to-device copy of
2 GiB, the reference dispatch for scaling the HBM byte counters.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

FP64_PEAK_TFLOPS = 78.6
HBM_PEAK_TBS = 8.0
GRID_SOURCES = ("paper_2608_30830_amd/csrc/kvr_grid.hip",
                "paper_2608_30830_amd/csrc/kvr_device.h",
                "paper_2608_30830_amd/csrc/kvr_internal.h")
COUNTERS_FILE = os.path.join(ROOT, "profiles", "grid_kernel_twotier-4096x64k_counters.txt")


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def grid_source_hash() -> str:
    h = hashlib.sha256()
    for rel in GRID_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def counter_traffic(workload: str, resamples: int):
    """HBM bytes per launch of the grid kernel from the committed counter
    summary, or None if it is for another workload or an older kernel."""
    if not os.path.exists(COUNTERS_FILE):
        return None
    kv = {}
    with open(COUNTERS_FILE) as fh:
        for line in fh:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("source_sha256") != grid_source_hash():
        return None
    if kv.get("workload") != workload or kv.get("resamples") != str(resamples):
        return None
    return float(kv["traffic_bytes_per_launch"])


class HipEvents:
    """Raw hipEvent_t handles (the library records them on its stream)."""

    def __init__(self, count: int):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.ev = []
        for _ in range(count):
            e = ctypes.c_void_p()
            if self.hip.hipEventCreate(ctypes.byref(e)) != 0:
                raise RuntimeError("hipEventCreate failed")
            self.ev.append(e)

    def elapsed_ms(self, a: int, b: int) -> float:
        ms = ctypes.c_float()
        if self.hip.hipEventElapsedTime(ctypes.byref(ms), self.ev[a], self.ev[b]) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(ms.value)

    def close(self):
        for e in self.ev:
            self.hip.hipEventDestroy(e)


def copy_calibration() -> int:
    import torch
    n = 1 << 28  # 2 GiB of float64
    x = torch.empty(n, dtype=torch.float64, device="cuda")
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": 8 * n, "copy_bytes_written": 8 * n}), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="twotier-4096x64k")
    ap.add_argument("--resamples", type=int, default=None,
                    help="truncate the bootstrap batch (for quick local runs)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=2,
                    help="bootstrap rows the CPU oracle evaluates for cpu_baseline")
    ap.add_argument("--paths", action="store_true",
                    help="also time the other entry points on their workloads")
    ap.add_argument("--table", action="store_true",
                    help="per-config table: GPU paths with their roofline fraction next to "
                         "the CPU oracle on one thread and on all threads, then exit")
    ap.add_argument("--replay-only", action="store_true",
                    help="time only the admission replay and the controller, then exit")
    ap.add_argument("--replay-reps", type=int, default=8192)
    ap.add_argument("--sort-scale", action="store_true",
                    help="time the SORTED path on 2^20, 2^22 and 2^24 waits, then exit")
    ap.add_argument("--copy-calibration", action="store_true")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1 "
                                   "(the bootstrap batch would shard by resample with no "
                                   "exchange; this build has no multi-GPU path)"}))
        return 2
    if args.copy_calibration:
        return copy_calibration()

    import torch

    import paper_2608_30830_amd as kvr
    import workloads

    if args.table:
        print(json.dumps({"table": results_table(kvr, workloads, torch)}), flush=True)
        return 0

    if args.sort_scale:
        print(json.dumps({"sort_scale": time_sort_scale(kvr, workloads, torch)}), flush=True)
        return 0

    if args.replay_only:
        print(json.dumps({"paths": time_replay(kvr, workloads, torch, args.replay_reps)}),
              flush=True)
        return 0

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

    log(f"[bench] warmup {args.warmup} step(s)")
    for _ in range(args.warmup):
        call.launch()
    torch.cuda.synchronize()
    st = call.status()
    if st != kvr.KVR_OK:
        raise kvr.KvrError(st, "warmup")

    log(f"[bench] timing {args.steps} step(s)")
    ev = HipEvents(2 * args.steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        kvr.kvr_set_profile_events(ev.ev[2 * i].value, ev.ev[2 * i + 1].value)
        call.launch()
    kvr.kvr_set_profile_events(None, None)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    st = call.status()
    if st != kvr.KVR_OK:
        raise kvr.KvrError(st, "timed steps")
    kern_ms = [ev.elapsed_ms(2 * i, 2 * i + 1) for i in range(args.steps)]
    ev.close()
    ms_per_step = 1000.0 * wall / args.steps
    kernel_ms = sum(kern_ms) / len(kern_ms)
    log(f"[bench] {ms_per_step:.1f} ms/step wall, grid kernel {kernel_ms:.1f} ms/launch")

    achieved = 2.0 * evals / (kernel_ms * 1e-3) / 1e12
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
                     "traffic": counter_traffic(args.workload, wl.n_resamples),
                     "kernel": "grid_kernel<32,1>", "kernel_ms": kernel_ms,
                     "flops_per_launch": 2.0 * evals},
    }

    if args.paths:
        out["paths"] = time_paths(kvr, workloads, torch)

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_rows)

    print(json.dumps(out), flush=True)
    return 0


def time_paths(kvr, workloads, torch):
    """Median milliseconds per call of the other entry points on their
    workloads (whole call, inputs resident)."""
    res = {}
    cases = (("weibull-1m", kvr.KVR_BRUTE), ("weibull-1m", kvr.KVR_SORTED),
             ("mix-64k", kvr.KVR_BRUTE), ("mix-64k", kvr.KVR_SORTED),
             ("tiny-exp-1k", kvr.KVR_BRUTE), ("tiny-exp-1k", kvr.KVR_SORTED),
             ("boot-1024x64k", None), ("boot-1024x64k", "factored"),
             ("twotier-4096x64k", "factored"))
    for name, method in cases:
        wl = workloads.make(name)
        pf = wl.platform
        pr = kvr.kvr_prices_from_platform(wl.kv_bytes_per_token, pf["hbm_usable_bytes"],
                                          pf["host_link_bytes_per_s"],
                                          pf["prefill_tokens_per_s"])
        g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
        w = torch.as_tensor(wl.wait_s).cuda()
        T = torch.as_tensor(wl.ctx_tokens).cuda()
        if method is None or method == "factored":
            call = kvr.BootstrapCall(w, T, torch.as_tensor(wl.idx).cuda(), pr, g,
                                     factored=method == "factored")
            run = call.launch
            key = f"{name}/{'factored' if method else 'bootstrap'}"
        else:
            out = torch.empty((wl.lam.size, wl.t1.size, wl.t2.size), dtype=torch.float64,
                              device="cuda")
            kvr.kvr_cost_grid(w, T, pr, g, method=method, out=out)

            def run(w=w, T=T, pr=pr, g=g, method=method, out=out):
                kvr.kvr_cost_grid(w, T, pr, g, method=method, out=out, check=False)
            key = f"{name}/{'sorted' if method == kvr.KVR_SORTED else 'brute'}"
        run()
        torch.cuda.synchronize()
        times = []
        for _ in range(7):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            run()
            b.record()
            torch.cuda.synchronize()
            times.append(a.elapsed_time(b))
        ms = sorted(times)[len(times) // 2]
        res[key] = {"ms": ms, "evaluations": wl.evaluations,
                    "evaluations_per_s": wl.evaluations / (ms * 1e-3)}
        log(f"[bench] path {key}: {ms:.3f} ms")
    res.update(time_platforms(kvr, workloads, torch))
    res.update(time_replay(kvr, workloads, torch))
    return res


# Algorithmic bytes per key of the SORTED path: eight digit passes, each an
# 8-byte histogram read, a 12-byte scatter read (key and payload) and a 12-byte
# write; key preparation (12 B read, 12 B written); the prefix scans (12 B read
# twice, 16 B written).
SORT_BYTES_PER_KEY = 8 * (8 + 12 + 12) + 24 + 40


def time_sort_scale(kvr, workloads, torch):
    """Median milliseconds per SORTED kvr_cost_grid call at 2^20, 2^22 and
    2^24 waits and the algorithmic bytes per second that implies."""
    res = {}
    for lg in (20, 22, 24):
        wl = workloads.sort_scale_case(lg)
        pf = wl.platform
        pr = kvr.kvr_prices_from_platform(wl.kv_bytes_per_token, pf["hbm_usable_bytes"],
                                          pf["host_link_bytes_per_s"],
                                          pf["prefill_tokens_per_s"])
        g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
        w = torch.as_tensor(wl.wait_s).cuda()
        T = torch.as_tensor(wl.ctx_tokens).cuda()
        out = torch.empty((wl.lam.size, wl.t1.size, wl.t2.size), dtype=torch.float64,
                          device="cuda")
        kvr.kvr_cost_grid(w, T, pr, g, method=kvr.KVR_SORTED, out=out)
        torch.cuda.synchronize()
        times = []
        for _ in range(9):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            kvr.kvr_cost_grid(w, T, pr, g, method=kvr.KVR_SORTED, out=out, check=False)
            b.record()
            torch.cuda.synchronize()
            times.append(a.elapsed_time(b))
        ms = sorted(times)[len(times) // 2]
        bps = SORT_BYTES_PER_KEY * wl.n / (ms * 1e-3)
        res[wl.name] = {"ms": ms, "keys_per_s": wl.n / (ms * 1e-3), "algorithmic_bytes_per_s": bps,
                        "hbm_frac": bps / (HBM_PEAK_TBS * 1e12)}
        log(f"[bench] sorted {wl.name}: {ms:.3f} ms, {bps / 1e12:.2f} TB/s algorithmic")
    return res


def time_platforms(kvr, workloads, torch):
    """The second workload: the three wait families as index rows, priced with
    each Table 3 vector; one kvr_bootstrap call per platform."""
    res = {}
    wl = workloads.cross_platform_case()
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    w = torch.as_tensor(wl.wait_s).cuda()
    T = torch.as_tensor(wl.ctx_tokens).cuda()
    idx = torch.as_tensor(wl.idx).cuda()
    for name, (a1, b2, b3) in workloads.PLATFORM_PRICES.items():
        pr = kvr.kvr_prices_from_platform(1.0, 1.0, 1.0, 1.0, 1.0, 425.0, 1800.0)
        pr.a1_per_token, pr.b2_per_token, pr.b3_per_token = a1, b2, b3
        call = kvr.BootstrapCall(w, T, idx, pr, g)
        call.launch()
        torch.cuda.synchronize()
        times = []
        for _ in range(7):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            call.launch()
            b.record()
            torch.cuda.synchronize()
            times.append(a.elapsed_time(b))
        ms = sorted(times)[len(times) // 2]
        key = f"{wl.name}-{name}/bootstrap"
        res[key] = {"ms": ms, "evaluations": wl.evaluations,
                    "evaluations_per_s": wl.evaluations / (ms * 1e-3)}
        log(f"[bench] path {key}: {ms:.3f} ms")
    return res


def time_replay(kvr, workloads, torch, reps: int = 8192):
    """The finite-capacity admission replay at 2 lambda_crit (the Table 6
    setting): ``reps`` sequences of 4,000 requests per wait family under the
    Eq. 3 timer, host-retain and the 10/30/60-minute timers."""
    res = {}
    lc = 425.0 / 1800.0
    pr = kvr.kvr_prices_from_platform(1.0, 1.0, 1.0, 1.0, 1.0, 425.0, 1800.0)
    pr.b2_per_token, pr.b3_per_token = 0.02, 1.91
    for family in workloads.FAMILIES:
        rc = workloads.replay_case(family, 2 * lc, reps=reps)
        t2 = [kvr.kvr_eq3_timer(pr, 2 * lc), float("inf"), 600.0, 1800.0, 3600.0]
        arr = torch.as_tensor(rc.arrival_s).cuda()
        w = torch.as_tensor(rc.wait_s).cuda()
        kvr.kvr_capacity_replay(arr, w, pr, t2)
        torch.cuda.synchronize()
        times = []
        for _ in range(5):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            kvr.kvr_capacity_replay(arr, w, pr, t2, check=False)
            b.record()
            torch.cuda.synchronize()
            times.append(a.elapsed_time(b))
        ms = sorted(times)[len(times) // 2]
        events = reps * len(t2) * rc.n
        key = f"replay-{family}-2x/{reps}x{rc.n}"
        res[key] = {"ms": ms, "replayed_requests": events,
                    "replayed_requests_per_s": events / (ms * 1e-3)}
        log(f"[bench] path {key}: {ms:.3f} ms")
    res.update(time_controller(kvr, workloads, torch, pr, reps))
    return res


def time_controller(kvr, workloads, torch, pr, reps: int):
    """The Section 3.4 controller calibrated at 2 lambda_crit on ``reps``
    sequences of 4,000 requests per wait family: both branches replayed,
    totals, frozen branch and P(W <= t*), all on the device."""
    res = {}
    lc = 425.0 / 1800.0
    pr.a1_per_token = 0.0176
    for family in workloads.FAMILIES:
        rc = workloads.replay_case(family, 2 * lc, reps=reps, seed=77)
        arr = torch.as_tensor(rc.arrival_s).cuda()
        w = torch.as_tensor(rc.wait_s).cuda()
        call = kvr.ControllerCall(arr, w, pr, 2 * lc)
        call.launch()
        out = call.result()
        times = []
        for _ in range(5):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            call.launch()
            b.record()
            torch.cuda.synchronize()
            times.append(a.elapsed_time(b))
        ms = sorted(times)[len(times) // 2]
        events = reps * 2 * rc.n
        key = f"controller-{family}-2x/{reps}x{rc.n}"
        res[key] = {"ms": ms, "replayed_requests": events,
                    "replayed_requests_per_s": events / (ms * 1e-3),
                    "branch": "expire" if out.branch == kvr.KVR_EXPIRE else "retain",
                    "p_short": out.p_short}
        log(f"[bench] path {key}: {ms:.3f} ms, branch {res[key]['branch']}, "
            f"P(W<=t*) {out.p_short:.4f}")
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


def _median_ms(torch, run, reps=5):
    run()
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        run()
        b.record()
        torch.cuda.synchronize()
        times.append(a.elapsed_time(b))
    return sorted(times)[len(times) // 2]


def results_table(kvr, workloads, torch, cpu_evals=2.0e9):
    """For each workload: whole-call GPU time of the brute-force path and of
    the closed form (SORTED for one sample, factored for bootstrap rows), the
    brute force's fraction of the fp64 peak (2 flop per evaluation), and the
    CPU oracle's rate on one thread and on every thread over a bounded
    sample (a prefix of the samples, or of one bootstrap row, holding about
    ``cpu_evals`` evaluations)."""
    import oracle
    all_threads = oracle.num_threads()
    rows = []
    for name in workloads.NAMES:
        wl = workloads.make(name)
        pf = wl.platform
        pr = kvr.kvr_prices_from_platform(wl.kv_bytes_per_token, pf["hbm_usable_bytes"],
                                          pf["host_link_bytes_per_s"],
                                          pf["prefill_tokens_per_s"])
        g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
        w = torch.as_tensor(wl.wait_s).cuda()
        T = torch.as_tensor(wl.ctx_tokens).cuda()
        reps = 3 if name.startswith("twotier") else 5
        if wl.idx is None:
            out = torch.empty((wl.lam.size, wl.t1.size, wl.t2.size), dtype=torch.float64,
                              device="cuda")
            brute = _median_ms(torch, lambda: kvr.kvr_cost_grid(w, T, pr, g, out=out,
                                                                check=False), reps)
            closed = _median_ms(torch, lambda: kvr.kvr_cost_grid(
                w, T, pr, g, method=kvr.KVR_SORTED, out=out, check=False), reps)
            closed_name = "sorted"
        else:
            idx = torch.as_tensor(wl.idx).cuda()
            bc = kvr.BootstrapCall(w, T, idx, pr, g)
            brute = _median_ms(torch, bc.launch, reps)
            fc = kvr.BootstrapCall(w, T, idx, pr, g, factored=True)
            closed = _median_ms(torch, fc.launch, reps)
            closed_name = "factored"
        evals = wl.evaluations
        per_sample = wl.t1.size * wl.t2.size * wl.lam.size
        m_cpu = int(max(1, min(wl.m, cpu_evals // per_sample)))
        op = oracle.workload_prices(wl)
        cpu = {}
        for threads in (1, all_threads):
            oracle.set_num_threads(threads)
            t0 = time.perf_counter()
            if wl.idx is None:
                oracle.cost_grid(wl.wait_s[:m_cpu], wl.ctx_tokens[:m_cpu], op, wl.t1, wl.t2,
                                 wl.lam)
            else:
                oracle.cost_grid(wl.wait_s, wl.ctx_tokens, op, wl.t1, wl.t2, wl.lam,
                                 idx_row=wl.idx[0][:m_cpu])
            cpu[threads] = m_cpu * per_sample / (time.perf_counter() - t0)
        oracle.set_num_threads(all_threads)
        row = {"workload": name, "evaluations": evals,
               "gpu_brute_ms": brute, "gpu_brute_evals_per_s": evals / (brute * 1e-3),
               "brute_fp64_frac": 2.0 * evals / (brute * 1e-3) / (FP64_PEAK_TFLOPS * 1e12),
               f"gpu_{closed_name}_ms": closed,
               "cpu_1_thread_evals_per_s": cpu[1],
               "cpu_all_threads_evals_per_s": cpu[all_threads], "cpu_threads": all_threads,
               "cpu_sample_evaluations": m_cpu * per_sample}
        rows.append(row)
        log(f"[bench] table {name}: brute {brute:.3f} ms ({row['brute_fp64_frac']:.3f} of fp64 "
            f"peak), {closed_name} {closed:.3f} ms, oracle {cpu[1]:.3e} / {cpu[all_threads]:.3e} "
            f"evaluations/s on 1 / {all_threads} threads")
    return rows


if __name__ == "__main__":
    sys.exit(main())
