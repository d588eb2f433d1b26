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
