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
    ap.add_argument("--cpu-rows", type=int, default=16,
                    help="bootstrap rows (evenly spaced, r = q * R / rows) the CPU oracle "
                         "evaluates for cpu_baseline")
    ap.add_argument("--cpu-draws", default="512,8192",
                    help="draws per row for the 1-thread and the all-thread oracle legs")
    ap.add_argument("--paths", action="store_true",
                    help="also time the other entry points on their workloads")
    ap.add_argument("--table", action="store_true",
                    help="per-config table: GPU paths with their roofline fraction next to "
                         "the CPU oracle on one thread and on all threads, then exit")
    ap.add_argument("--replay-only", action="store_true",
                    help="time only the admission replay and the controller, then exit")
    ap.add_argument("--replay-reps", type=int, default=8192)
    ap.add_argument("--factored-only", action="store_true",
                    help="time only kvr_bootstrap_factored on the bootstrap workloads, then exit")
    ap.add_argument("--sort-scale", action="store_true",
                    help="time the SORTED path on 2^20, 2^22, 2^23 and 2^24 waits, then exit")
    ap.add_argument("--copy-calibration", action="store_true")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "kvr runs on one GPU only; --gpus must be 1 (the "
                                   "bootstrap batch would shard by resample with no exchange; "
                                   "there is no multi-GPU path)"}))
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

    if args.factored_only:
        print(json.dumps({"paths": time_factored(kvr, workloads, torch)}), flush=True)
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
    inputs = {"wait_s_sha256": sha256_of(wl.wait_s), "ctx_tokens_sha256": sha256_of(wl.ctx_tokens),
              "idx_sha256": sha256_of(wl.idx)}
    hbm_copy = copy_rate(torch)

    log(f"[bench] warmup {args.warmup} step(s)")
    for _ in range(args.warmup):
        call.launch()
    torch.cuda.synchronize()
    st = call.status()
    if st != kvr.KVR_OK:
        raise kvr.KvrError(st, "warmup")

    log(f"[bench] timing {args.steps} step(s)")
    ev = HipEvents(2 * args.steps)
    clock = ClockSampler()
    torch.cuda.synchronize()
    clock.start()
    t0 = time.perf_counter()
    for i in range(args.steps):
        kvr.kvr_set_profile_events(ev.ev[2 * i].value, ev.ev[2 * i + 1].value)
        call.launch()
    kvr.kvr_set_profile_events(None, None)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    clock.stop()
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
                   "evaluations_per_step": evals, "method": "brute-force grid: one fp64 FMA per (draw, policy, load) for "
                             "the load-dependent holding term; load-independent terms per "
                             "(draw, t1) and recompute counts per (draw, deadline) through "
                             "deadline bins; selection fused"},
        "roofline": {"bound": "alu", "achieved": achieved, "peak": FP64_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / FP64_PEAK_TFLOPS,
                     "traffic": counter_traffic(args.workload, wl.n_resamples),
                     "kernel": "grid_kernel<32,1>", "kernel_ms": kernel_ms,
                     "flops_per_launch": 2.0 * evals},
        "inputs": inputs,
        "gpu_sclk_mhz": clock.summary(),
        "hbm_copy": hbm_copy,
    }

    if args.paths:
        out["paths"] = time_paths(kvr, workloads, torch)

    if not args.no_cpu_baseline:
        draws = [int(x) for x in args.cpu_draws.split(",")]
        out["cpu_baseline"], out["parity"] = cpu_leg(wl, args.cpu_rows, draws,
                                                     call.best.cpu().numpy(),
                                                     call.best_cost.cpu().numpy())

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
            call = kvr.CostGridCall(w, T, pr, g, method=method)
            run = call.launch
            key = f"{name}/{'sorted' if method == kvr.KVR_SORTED else 'brute'}"
        ms = _median_ms(torch, run, 11)
        res[key] = {"ms": ms, "evaluations": wl.evaluations,
                    "evaluations_per_s": wl.evaluations / (ms * 1e-3)}
        log(f"[bench] path {key}: {ms:.3f} ms")
    res.update(time_platforms(kvr, workloads, torch))
    res.update(time_replay(kvr, workloads, torch))
    return res


# Algorithmic bytes per key of the SORTED path (no order requested): the first
# digit's tile histograms from the waits (8 B read); the histograms of the
# other seven digits (below 2^22 keys each reads the 8-byte keys; from 2^22 the
# one-byte digits that the previous scatter wrote: 1 B read, and 1 B written
# by each of the first seven scatters); eight scatters (12 B read, 12 B
# written each; the first reads the waits and context sizes); the tile and
# 64-key chunk sums (12 B read, 16 B written per 64 keys).  The closed form
# then reads N and S at its query positions only.
SORT_DIGIT_BYTES_FROM = 1 << 22


def sort_bytes_per_key(n: int) -> float:
    hist = 7 * (1 + 1) if n >= SORT_DIGIT_BYTES_FROM else 7 * 8
    return 8 + hist + 8 * 24 + 12 + 16 / 64


def time_factored(kvr, workloads, torch):
    """kvr_bootstrap_factored on boot-1024x64k and twotier-4096x64k (median of
    eleven calls after about 100 ms of calls, inputs resident)."""
    res = {}
    for name in ("boot-1024x64k", "twotier-4096x64k"):
        wl = workloads.make(name)
        pf = wl.platform
        pr = kvr.kvr_prices_from_platform(wl.kv_bytes_per_token, pf["hbm_usable_bytes"],
                                          pf["host_link_bytes_per_s"],
                                          pf["prefill_tokens_per_s"])
        g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
        call = kvr.BootstrapCall(torch.as_tensor(wl.wait_s).cuda(),
                                 torch.as_tensor(wl.ctx_tokens).cuda(),
                                 torch.as_tensor(wl.idx).cuda(), pr, g, factored=True)
        ms = _median_ms(torch, call.launch, 11)
        key = f"{name}/factored"
        res[key] = {"ms": ms}
        log(f"[bench] path {key}: {ms:.3f} ms")
    return res


def time_sort_scale(kvr, workloads, torch):
    """Median milliseconds per SORTED kvr_cost_grid call at 2^20, 2^22, 2^23
    and 2^24 waits and the algorithmic bytes per second that implies."""
    res = {}
    for lg in (20, 22, 23, 24):
        wl = workloads.sort_scale_case(lg)
        pf = wl.platform
        pr = kvr.kvr_prices_from_platform(wl.kv_bytes_per_token, pf["hbm_usable_bytes"],
                                          pf["host_link_bytes_per_s"],
                                          pf["prefill_tokens_per_s"])
        g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
        w = torch.as_tensor(wl.wait_s).cuda()
        T = torch.as_tensor(wl.ctx_tokens).cuda()
        call = kvr.CostGridCall(w, T, pr, g, method=kvr.KVR_SORTED)
        ms = _median_ms(torch, call.launch, 11)
        bps = sort_bytes_per_key(wl.n) * wl.n / (ms * 1e-3)
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
        ms = _median_ms(torch, call.launch, 11)
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
        kvr.kvr_capacity_replay(arr, w, pr, t2)   # checked once
        ms = _median_ms(torch, lambda: kvr.kvr_capacity_replay(arr, w, pr, t2, check=False), 11)
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
        ms = _median_ms(torch, call.launch, 11)
        events = reps * 2 * rc.n
        key = f"controller-{family}-2x/{reps}x{rc.n}"
        res[key] = {"ms": ms, "replayed_requests": events,
                    "replayed_requests_per_s": events / (ms * 1e-3),
                    "branch": "expire" if out.branch == kvr.KVR_EXPIRE else "retain",
                    "p_short": out.p_short}
        log(f"[bench] path {key}: {ms:.3f} ms, branch {res[key]['branch']}, "
            f"P(W<=t*) {out.p_short:.4f}")
    return res


def sha256_of(arr) -> str:
    import numpy as np
    return hashlib.sha256(np.ascontiguousarray(arr).tobytes()).hexdigest()


def copy_rate(torch):
    """A plain 2 GiB device-to-device copy (median of 5, torch events): the
    practical HBM ceiling of this machine, read + write bytes per second."""
    n = 1 << 28
    x = torch.empty(n, dtype=torch.float64, device="cuda")
    y = torch.empty_like(x)
    ms = _median_ms(torch, lambda: y.copy_(x), 5)
    del x, y
    torch.cuda.empty_cache()
    return {"bytes": 2 * 8 * n, "ms": ms, "tbps": 2 * 8 * n / (ms * 1e-3) / 1e12,
            "frac_of_peak": 2 * 8 * n / (ms * 1e-3) / (HBM_PEAK_TBS * 1e12)}


class ClockSampler:
    """Samples the GPU's current shader clock (the starred level of the
    driver's pp_dpm_sclk table) every 0.25 s while the timed steps run."""

    def __init__(self):
        import glob
        files = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
        self.path = files[0] if files else None
        self.samples = []
        self._stop = None

    def _read(self):
        try:
            with open(self.path) as fh:
                for line in fh:
                    if "*" in line:
                        return float(line.split(":")[1].strip().split("Mhz")[0].split("MHz")[0])
        except (OSError, ValueError, IndexError):
            return None
        return None

    def start(self):
        if self.path is None:
            return
        import threading
        self._stop = threading.Event()

        def loop():
            while not self._stop.wait(0.25):
                v = self._read()
                if v is not None:
                    self.samples.append(v)
        self._thread = threading.Thread(target=loop, daemon=True)
        self._thread.start()

    def stop(self):
        if self._stop is not None:
            self._stop.set()
            self._thread.join()

    def summary(self):
        if not self.samples:
            return None
        s = sorted(self.samples)
        return {"samples": len(s), "min": s[0], "median": s[len(s) // 2], "max": s[-1],
                "source": "pp_dpm_sclk, every 0.25 s during the timed steps"}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_leg(wl, rows: int, draws, gpu_best, gpu_best_cost):
    """The cpu_baseline leg.  (1) The oracle's double loop, as it stands, on a
    bounded sample of the same workload: ``rows`` evenly spaced bootstrap rows
    (r = q * R / rows), each cut to its first draws (draws[0] on one thread,
    draws[1] on every thread), every policy and load; the rate is extrapolated
    linearly in evaluations to the whole workload.  (2) A parity sample of the
    timed call: the GPU's selections and best costs on the same rows (full
    length) against the oracle's closed form."""
    import numpy as np
    import oracle
    pr = oracle.workload_prices(wl)
    R = wl.n_resamples
    sel = sorted({(q * R) // rows for q in range(rows)}) if wl.idx is not None else [None]
    per_draw = wl.t1.size * wl.t2.size * wl.lam.size
    all_threads = oracle.num_threads()
    legs = {}
    for threads, cut in ((1, draws[0]), (all_threads, draws[1])):
        cut = min(cut, wl.m)
        oracle.set_num_threads(threads)
        log(f"[bench] cpu baseline: oracle on {len(sel)} row(s) x {cut} draws, {threads} thread(s)")
        t0 = time.perf_counter()
        for r in sel:
            if r is None:
                oracle.cost_grid(wl.wait_s[:cut], wl.ctx_tokens[:cut], pr, wl.t1, wl.t2, wl.lam)
            else:
                oracle.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                 idx_row=wl.idx[r][:cut])
        dt = time.perf_counter() - t0
        ev = len(sel) * cut * per_draw
        legs[threads] = {"value": ev / dt, "cores": threads, "seconds": dt, "evaluations": ev,
                         "draws_per_row": cut,
                         "whole_workload_seconds": wl.evaluations / (ev / dt)}
    oracle.set_num_threads(all_threads)
    rows_txt = (f"rows r = q * {R // rows} (q = 0..{len(sel) - 1}) of {R}" if wl.idx is not None
                else "a prefix of the sample")
    base = dict(legs[all_threads])
    base.update({
        "unit": "evaluations/s", "kind": "oracle",
        "sample": f"{rows_txt}, first {legs[all_threads]['draws_per_row']} draws of each "
                  f"(all threads) / first {legs[1]['draws_per_row']} (one thread), every "
                  f"policy and load",
        "single_thread": legs[1], "all_threads": legs[all_threads],
        "extrapolated": True,
        "extrapolation": "linear in evaluations: whole-workload seconds = evaluations per step "
                         "/ measured rate",
        "cpu_model": cpu_model(), "os_cpu_count": os.cpu_count(),
        "affinity_cpus": len(os.sched_getaffinity(0)),
    })
    # parity sample of the timed call on the same rows, full length
    parity = {"reference": "oracle closed form (sorted prefix sums), full rows",
              "rows": [r for r in sel if r is not None]}
    if wl.idx is not None:
        mism, near, err, gap = 0, 0, 0.0, float("inf")
        for r in sel:
            ref = oracle.closed_form_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                          idx_row=wl.idx[r])
            rb, rbc, _ = oracle.select(ref, wl.t2)
            err = max(err, float(np.max(np.abs(gpu_best_cost[r] - rbc) / np.abs(rbc))))
            flat = ref.reshape(ref.shape[0], -1)
            for l in range(flat.shape[0]):
                if gpu_best[r, l] != rb[l]:
                    c_gpu, c_ref = flat[l, gpu_best[r, l]], flat[l, rb[l]]
                    if abs(c_gpu - c_ref) <= 1e-11 * abs(c_ref):
                        near += 1
                    else:
                        mism += 1
                row = np.sort(flat[l])
                higher = row[row > row[0]]
                if higher.size and row[0] != 0:
                    gap = min(gap, float((higher[0] - row[0]) / abs(row[0])))
        parity.update({"index_mismatches": mism, "near_tie_picks": near,
                       "max_rel_err_best_cost": err, "min_runner_up_gap": gap})
        log(f"[bench] parity on {len(sel)} rows: {mism} mismatches, {near} near ties, "
            f"max rel err {err:.2e}, smallest runner-up gap {gap:.2e}")
    return base, parity


def _warm(torch, run, ms=100.0):
    """Runs ``run`` back to back for about ``ms`` of wall time, so that the
    timed calls that follow see the clock a busy GPU runs at (a few short
    calls after an idle spell are timed while the clock is still rising)."""
    t0 = time.perf_counter()
    run()
    torch.cuda.synchronize()
    while (time.perf_counter() - t0) * 1e3 < ms:
        run()
        torch.cuda.synchronize()


def _median_ms(torch, run, reps=5):
    _warm(torch, run)
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
        reps = 3 if name.startswith("twotier") else 11
        if wl.idx is None:
            brute = _median_ms(torch, kvr.CostGridCall(w, T, pr, g).launch, reps)
            closed = _median_ms(torch, kvr.CostGridCall(w, T, pr, g, method=kvr.KVR_SORTED).launch,
                                reps)
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
