"""Pins of the seeded inputs (no GPU): every array that the tests, the smoke
check and the benchmark draw from workloads.py hashes to the SHA-256 recorded
in tests/golden/input_hashes.txt.  A change in numpy's generators or in a
recipe (the Section 4.1 wait families, the context sizes, the bootstrap rows,
the Poisson arrivals) fails here first, instead of silently moving a seeded
pin such as the tiny workload's memoryless selection."""
import importlib.util
import os

from tests import helpers as H

SPEC = importlib.util.spec_from_file_location(
    "make_input_hashes", os.path.join(H.GOLDEN, "make_input_hashes.py"))
gen = importlib.util.module_from_spec(SPEC)
SPEC.loader.exec_module(gen)


def _recorded():
    out = {}
    for row in H.read_table("input_hashes.txt"):
        name, field, digest, shape = row
        out[(name, field)] = (digest, shape)
    return out


def test_every_seeded_input_matches_its_recorded_hash():
    rec = _recorded()
    seen = set()
    for name, field, arr in gen.entries():
        key = (name, field)
        assert key in rec, f"no recorded hash for {key}"
        digest, shape = rec[key]
        assert "x".join(map(str, arr.shape)) == shape, key
        assert gen.sha(arr) == digest, f"{name} {field}: inputs changed"
        seen.add(key)
    assert seen == set(rec)


def test_recorded_hashes_cover_every_workload():
    names = {k[0] for k in _recorded()}
    import workloads
    assert set(workloads.NAMES) <= names
    for fam in workloads.FAMILIES:
        assert f"replay-{fam}-2x" in names and f"calibration-{fam}-2x" in names
