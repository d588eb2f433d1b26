"""Writes input_hashes.txt: SHA-256 of every seeded input array that the
tests, the smoke check and the benchmark draw from workloads.py (little-endian
bytes of the arrays as generated).  Run from the repository root:
    python tests/golden/make_input_hashes.py
It calls only workloads.py (which draws numbers and lays out grids; neither the
library nor the oracle is involved)."""
import hashlib
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import workloads  # noqa: E402


def sha(a):
    a = np.ascontiguousarray(a)
    assert a.dtype.byteorder in ("<", "=", "|")
    return hashlib.sha256(a.tobytes()).hexdigest()


def entries():
    for name in workloads.NAMES:
        wl = workloads.make(name)
        yield name, "wait_s", wl.wait_s
        yield name, "ctx_tokens", wl.ctx_tokens
        yield name, "grid", np.concatenate([wl.t1, wl.t2, wl.lam])
        if wl.idx is not None:
            yield name, "idx_first_row", wl.idx[0]
            yield name, "idx_last_row", wl.idx[-1]
            yield name, "idx", wl.idx
    for lg in (20, 24):
        wl = workloads.sort_scale_case(lg)
        yield wl.name, "wait_s", wl.wait_s
        yield wl.name, "ctx_tokens", wl.ctx_tokens
    wl = workloads.cross_platform_case()
    yield wl.name, "wait_s", wl.wait_s
    yield wl.name, "grid", np.concatenate([wl.t1, wl.t2, wl.lam])
    lc = 425.0 / 1800.0
    for family in workloads.FAMILIES:
        rc = workloads.replay_case(family, 2 * lc, reps=4)
        yield f"replay-{family}-2x", "arrival_s", rc.arrival_s
        yield f"replay-{family}-2x", "wait_s", rc.wait_s
        rc = workloads.replay_case(family, 2 * lc, reps=4, seed=77)
        yield f"calibration-{family}-2x", "wait_s", rc.wait_s


def main():
    lines = ["# SHA-256 of the seeded inputs (workloads.py); written by make_input_hashes.py",
             "# workload field sha256 shape"]
    for name, field, arr in entries():
        lines.append(f"{name} {field} {sha(arr)} {'x'.join(map(str, np.shape(arr)))}")
    with open(os.path.join(HERE, "input_hashes.txt"), "w") as fh:
        fh.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()
