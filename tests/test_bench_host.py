"""Host-side behaviour of bench.py that needs no GPU: the one-GPU guard and the
rule that HBM traffic is reported only from a counter summary taken on the
current grid-kernel sources and the same workload."""
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_traffic_only_for_matching_sources_and_workload(tmp_path, monkeypatch):
    summary = tmp_path / "counters.txt"
    summary.write_text("# header\nworkload: twotier-4096x64k\nresamples: 4096\n"
                       "traffic_bytes_per_launch: 2.5e+09\n"
                       f"source_sha256: {bench.grid_source_hash()}\n")
    monkeypatch.setattr(bench, "COUNTERS_FILE", str(summary))
    assert bench.counter_traffic("twotier-4096x64k", 4096) == 2.5e9
    assert bench.counter_traffic("twotier-4096x64k", 8) is None       # a truncated batch
    assert bench.counter_traffic("boot-1024x64k", 4096) is None       # another workload
    summary.write_text(summary.read_text().replace(bench.grid_source_hash(), "0" * 64))
    assert bench.counter_traffic("twotier-4096x64k", 4096) is None    # an older kernel
    monkeypatch.setattr(bench, "COUNTERS_FILE", str(tmp_path / "missing.txt"))
    assert bench.counter_traffic("twotier-4096x64k", 4096) is None


def test_grid_hash_covers_the_kernel_sources():
    for rel in bench.GRID_SOURCES:
        assert os.path.exists(os.path.join(ROOT, rel)), rel
    assert "paper_2608_30830_amd/csrc/kvr_grid.hip" in bench.GRID_SOURCES


def test_cpu_leg_reports_both_legs_and_a_parity_sample():
    """cpu_baseline: a one-thread and an all-thread leg on evenly spaced rows,
    extrapolated linearly, with the CPU model; the parity sample compares the
    selections handed to it (here the oracle's own) with the closed form."""
    import oracle
    import workloads
    wl = workloads.make("twotier-4096x64k", resamples=32)
    pr = oracle.workload_prices(wl)
    best, bc = oracle.closed_form_bootstrap(wl.wait_s, wl.ctx_tokens, wl.idx, pr, wl.t1, wl.t2,
                                            wl.lam)
    base, parity = bench.cpu_leg(wl, 16, [4, 16], best, bc)
    assert base["kind"] == "oracle" and base["extrapolated"] is True
    assert base["single_thread"]["cores"] == 1 and base["single_thread"]["draws_per_row"] == 4
    assert base["cores"] == oracle.num_threads() and base["all_threads"]["draws_per_row"] == 16
    assert base["value"] == base["all_threads"]["value"] > 0
    assert base["all_threads"]["evaluations"] == 16 * 16 * 64 * 257 * 32
    assert base["cpu_model"] and base["os_cpu_count"] >= 1
    assert parity["rows"] == list(range(0, 32, 2))
    assert parity["index_mismatches"] == 0 and parity["max_rel_err_best_cost"] == 0.0
