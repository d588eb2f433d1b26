"""A seeded sweep of grid shapes through every grid entry point against the
oracle's double loop: the policy count below, at and off multiples of the
64-lane groups, one to several load tiles (up to 40 loads), single samples
and bootstrap rows of every length, sample splits and fused selection,
duplicated waits and waits sitting on timers; every fourth case charges the
copy at offload.  Costs within 1e-9 relative,
selections identical up to rounding-level near ties."""
import numpy as np
import pytest

import workloads
from tests.test_gpu_parity import (_dev, _f64, _i32, _lib_prices, _np, assert_costs,
                                   assert_selection)

pytestmark = pytest.mark.gpu


def _shape(i):
    rng = np.random.Generator(np.random.PCG64(5000 + i))
    k1 = int(rng.choice([1, 1, 2, 3, 5]))
    k2 = int(rng.choice([2, 9, 33, 63, 64, 65, 127, 128, 200]))
    L = int(rng.choice([1, 3, 4, 5, 8, 16, 17, 31, 32, 40]))
    n = int(rng.choice([1, 7, 64, 129, 1000, 5000, 20000]))
    R = int(rng.choice([0, 0, 1, 2, 3, 7]))
    m = None if R == 0 else int(rng.choice([1, 100, n, 3000]))
    return 6000 + i, n, k1, k2, L, R, m


CASES = [_shape(i) for i in range(40)]


@pytest.fixture(scope="module")
def kvr():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2608_30830_amd as k
    k.load_library()
    return k


@pytest.mark.parametrize("case", CASES, ids=[f"s{c[0]}-n{c[1]}-k{c[2]}x{c[3]}-L{c[4]}-R{c[5]}"
                                             for c in CASES])
def test_grid_shapes(kvr, oracle_mod, case):
    seed, n, k1, k2, L, R, m = case
    wl = workloads.random_case(seed, n, k1, k2, L, resamples=R, m=m, ties=True,
                               inf_last=(seed % 3 != 0))
    pr = oracle_mod.workload_prices(wl)
    lp = _lib_prices(kvr, wl)
    if seed % 4 == 1:   # the optional charge for the copy at offload, on both sides
        pr.boff = pr.b2
        lp.offload_per_token = lp.b2_per_token
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    w, T = _dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32())
    if wl.idx is None:
        ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam)
        rb = oracle_mod.select(ref, wl.t2)[0]
        for method in (kvr.KVR_BRUTE, kvr.KVR_SORTED):
            cost = kvr.kvr_cost_grid(w, T, lp, g, method=method)
            assert_costs(_np(cost), ref)
            best = kvr.kvr_select_policy(cost, g.last_inf)[0]
            assert_selection(ref, _np(best), rb)
        return
    idx = _dev(wl.idx, _i32())
    for factored in (False, True):
        best, bc, cost = kvr.kvr_bootstrap(w, T, idx, lp, g, want_cost=True, factored=factored)
        for r in range(wl.n_resamples):
            ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                       idx_row=wl.idx[r])
            assert_costs(_np(cost)[r], ref)
            rb, rbc, _ = oracle_mod.select(ref, wl.t2)
            assert_selection(ref, _np(best)[r], rb)
            assert_costs(_np(bc)[r], rbc)


@pytest.mark.parametrize("n", [2047, 2048, 2049, 4096, 4097, 262143, 262144, 300001, 524288])
def test_sort_path_boundaries(kvr, oracle_mod, n):
    """Sample sizes around the one-block sort (at most 2,048 waits), around the
    tile sizes of the multi-block sort (512-key tiles below 2^18 waits, 1,024
    below 2^19, 2,048 from there) and a ragged last tile: the SORTED grid and
    its order against the oracle, and the factored bootstrap, which sorts the
    same way."""
    wl = workloads.random_case(7000 + n, n, 2, 70, 5, resamples=2, m=n, ties=True)
    pr = oracle_mod.workload_prices(wl)
    lp = _lib_prices(kvr, wl)
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    w, T = _dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32())
    cost, perm = kvr.kvr_cost_grid(w, T, lp, g, method=kvr.KVR_SORTED, want_perm=True)
    assert np.array_equal(_np(perm), oracle_mod.stable_order(wl.wait_s))
    ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam)
    assert_costs(_np(cost), ref)
    best, bc, cost = kvr.kvr_bootstrap(w, T, _dev(wl.idx, _i32()), lp, g, want_cost=True,
                                       factored=True)
    for r in range(2):
        ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                   idx_row=wl.idx[r])
        assert_costs(_np(cost)[r], ref)
        rb = oracle_mod.select(ref, wl.t2)[0]
        assert_selection(ref, _np(best)[r], rb)
