"""The one-launch small-sample brute force (kvr_cost_grid, BRUTE, one sample
within the small-sample limits): sample split groups below, at and off the
batches of eight that the launch adds up, several load tiles, eight t1 timers,
no finite deadline, the largest pre-pass histogram and the most pre-pass blocks
and (group, load tile)s the path takes (and one grid past that limit), and a
workspace that holds another call's counters and partials; costs against the
oracle's double loop within 1e-9 relative."""
import numpy as np
import pytest

import workloads
from tests.test_gpu_parity import _dev, _f64, _i32, _lib_prices, _np, assert_costs

pytestmark = pytest.mark.gpu

# name, n, t1 timers, t2 timers, loads, infinite last t2, seed
CASES = [
    ("groups1-t1x8-tiles", 1000, 8, 64, 40, True, 71),      # 512 policies, one split group
    ("groups13", 13312, 1, 2, 4, True, 72),                 # 104 splits: batches of 8 and 5
    ("groups64", 65536, 1, 8, 3, True, 73),                 # 512 splits: eight full batches
    ("tiles", 5000, 3, 100, 70, True, 74),
    ("no-finite-deadline", 4000, 2, 1, 5, True, 75),        # t2 = [inf]: no recompute bins
    ("histogram-64x1024", 65536, 4, 256, 2, False, 76),     # 64 pre-pass rows of 1,024 bins
    ("prepass-256-blocks", 262144, 1, 200, 40, True, 77),   # the most pre-pass blocks, 256
    ("group-tiles-4096", 100, 8, 512, 2048, True, 78),      # 64 groups x 64 tiles of 32 loads
    ("group-tiles-4160", 100, 8, 512, 2080, True, 79),      # 65 tiles: past the limit, the multi-launch path
]


@pytest.fixture(scope="module")
def kvr():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2608_30830_amd as k
    k.load_library()
    return k


def _case(kvr, oracle_mod, name, n, k1, k2, L, inf_last, seed):
    # waits planted on deadlines need a finite one
    wl = workloads.random_case(seed, n, k1, k2, L, inf_last=inf_last,
                               ties=not (inf_last and k2 == 1))
    ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, oracle_mod.workload_prices(wl),
                               wl.t1, wl.t2, wl.lam)
    return wl, ref


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_small_path_against_oracle(kvr, oracle_mod, case):
    wl, ref = _case(kvr, oracle_mod, *case)
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    cost = kvr.kvr_cost_grid(_dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32()),
                             _lib_prices(kvr, wl), g, method=kvr.KVR_BRUTE)
    assert_costs(_np(cost), ref)


def test_small_path_stale_workspace(kvr, oracle_mod):
    """One workspace, first filled with 0xff bytes, then reused by calls of
    other shapes in a row: every call clears its own counters."""
    import torch
    ws = torch.full((64 << 20,), 0xff, dtype=torch.uint8, device="cuda")
    for case in (CASES[2], CASES[1], CASES[0], CASES[1]):
        wl, ref = _case(kvr, oracle_mod, *case)
        g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
        cost = kvr.kvr_cost_grid(_dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32()),
                                 _lib_prices(kvr, wl), g, method=kvr.KVR_BRUTE, workspace=ws)
        assert_costs(_np(cost), ref)
