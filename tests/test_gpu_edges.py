"""GPU parity on the edges that the stable order and the fused selection promise.

* Waits that mix -0.0, +0.0 and repeated positive values.  The stable order
  (Section 3.4's replay only needs the waits in order; ties keep input order)
  treats -0.0 as +0.0.  They run through the one-block sort (n <= 2,048), the
  multi-block sort at each of its tile sizes, the brute force, the bootstrap
  and the factored bootstrap.  The order is compared bit for bit, costs within
  1e-9 relative.
* The fused arg-min of kvr_bootstrap (a per-wave candidate per load, then one
  reduction per resample) in every lane mapping: fewer than 64 host timers
  (one policy per lane), a policy count that is a multiple of 64, a policy
  count that lets a wave straddle two resamples, and a grid of at least 32,768
  base waves.  Its picks must equal the selection rule (cost ascending, exact
  ties to the larger flat index) applied to the GPU's own cost tensor, exactly.
* Load tiles of 16, 8 and 4 loads on grids whose 64-lane groups straddle t1
  rows or resamples, fused and split, through kvr_bootstrap and kvr_cost_grid
  (above the small-sample path), against the oracle's double loop.
* The full two-tier cost tensor (64 x 257 x 32 policies and loads) of fixed
  rows of the 4,096-row bench workload, from the bench's own launch, against
  the oracle's double loop element by element.
"""
import numpy as np
import pytest

import workloads
from tests import helpers as H
from tests.test_gpu_parity import (RTOL, TIE_RTOL, _dev, _f64, _i32, _lib_prices, _np,
                                   assert_costs, assert_selection)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kvr():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2608_30830_amd as k
    k.load_library()
    return k


def signed_zero_case(seed, n, k1, k2, L, resamples=2, neg_t1=False):
    """A random case whose waits hold -0.0 and +0.0 (an eighth each, the two
    interleaved), runs of one repeated positive wait, and waits equal to t1
    values; optional t1 = -0.0 (a valid t1 >= 0)."""
    wl = workloads.random_case(seed, n, k1, k2, L, resamples=resamples, ties=True)
    rng = np.random.Generator(np.random.PCG64(seed + 7))
    w = wl.wait_s.copy()
    pos = rng.permutation(n)
    q = max(1, n // 8)
    w[pos[:q]] = -0.0
    w[pos[q:2 * q]] = 0.0
    w[pos[2 * q:3 * q]] = w[pos[-1]] if w[pos[-1]] > 0 else 17.0
    w[pos[3 * q:3 * q + 3]] = wl.t1[-1]
    wl.wait_s = w
    if neg_t1:
        wl.t1 = wl.t1.copy()
        wl.t1[0] = -0.0
    return wl


# n <= 2,048 takes the one-block sort; above it the multi-block sort with
# tiles of 512 keys (n < 2^18), 1,024 keys (n < 2^19) and 2,048 keys
SIGNED_ZERO_SIZES = [(401, 700, 2, 9, 3), (402, 2048, 1, 70, 5), (403, 2049, 3, 66, 4),
                     (404, 70000, 2, 65, 6), (405, 300000, 1, 40, 3), (406, 600000, 2, 20, 3)]


@pytest.mark.parametrize("case", SIGNED_ZERO_SIZES, ids=[f"n{c[1]}" for c in SIGNED_ZERO_SIZES])
def test_signed_zero_waits_every_path(kvr, oracle_mod, case):
    seed, n, k1, k2, L = case
    wl = signed_zero_case(seed, n, k1, k2, L, neg_t1=(seed % 2 == 0))
    assert np.signbit(wl.wait_s).sum() >= n // 8 and (wl.wait_s == 0).sum() >= n // 4
    pr = oracle_mod.workload_prices(wl)
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    lp = _lib_prices(kvr, wl)
    w, T = _dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32())
    import torch
    assert torch.signbit(w).sum().item() == np.signbit(wl.wait_s).sum()   # -0.0 reached the GPU
    ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam)
    rb = oracle_mod.select(ref, wl.t2)[0]
    ref_perm = oracle_mod.stable_order(wl.wait_s)
    # the stable order ranks -0.0 and +0.0 as one value, in input order
    zeros = np.nonzero(wl.wait_s == 0)[0]
    assert np.array_equal(ref_perm[:zeros.size], zeros)
    brute = kvr.kvr_cost_grid(w, T, lp, g, method=kvr.KVR_BRUTE)
    sorted_cost, perm = kvr.kvr_cost_grid(w, T, lp, g, method=kvr.KVR_SORTED, want_perm=True)
    assert np.array_equal(_np(perm), ref_perm)
    for c in (brute, sorted_cost):
        assert_costs(_np(c), ref)
        assert_selection(ref, _np(kvr.kvr_select_policy(c, g.last_inf)[0]), rb)
    idx = _dev(wl.idx, _i32())
    for factored in (False, True):
        best, bc, cost = kvr.kvr_bootstrap(w, T, idx, lp, g, want_cost=True, factored=factored)
        for r in range(wl.n_resamples):
            rr = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                      idx_row=wl.idx[r])
            assert_costs(_np(cost)[r], rr)
            rsel, rbc, _ = oracle_mod.select(rr, wl.t2)
            assert_selection(rr, _np(best)[r], rsel)
            assert_costs(_np(bc)[r], rbc)


def test_signed_zero_crossover_and_replay(kvr, oracle_mod):
    """-0.0 waits count as waits at or below t* and resume at their arrival."""
    rc = workloads.replay_case("mixture", 2.0 * 425.0 / 1800.0, reps=3, n=1500, seed=41)
    w = rc.wait_s.copy()
    w[:, ::5] = -0.0
    w[:, 1::5] = 0.0
    pf = workloads.PLATFORM
    lp = kvr.kvr_prices_from_platform(1.0, 1.0, 1.0, 1.0, 1.0, pf["host_slots_c2"],
                                      pf["w_ref_s"])
    lp.a1_per_token, lp.b2_per_token, lp.b3_per_token = workloads.PLATFORM_PRICES["h100-nvl"]
    a1, b2, b3 = workloads.PLATFORM_PRICES["h100-nvl"]
    count, frac = kvr.kvr_crossover_statistic(_dev(w.ravel(), _f64()), lp)
    assert int(_np(count)[0]) == oracle_mod.crossover_count(w, a1, b3)
    t2 = [60.0, 600.0, float("inf")]
    cost, rest, _ = kvr.kvr_capacity_replay(_dev(rc.arrival_s, _f64()), _dev(w, _f64()), lp, t2)
    ref_cost, ref_rest = oracle_mod.capacity_replay_batch(rc.arrival_s, w, 425, t2, b2, b3)
    assert np.array_equal(_np(rest), ref_rest)
    assert_costs(_np(cost), ref_cost, rtol=1e-12)


def _fused_plan_cases():
    # (seed, n, K1, K2, L, R, m): m <= 1,023 keeps every resample in one
    # split, so kvr_bootstrap selects inside the grid kernel
    return {
        "per-lane": (411, 900, 3, 9, 5, 7, 1000),          # K2 < 64
        "rows1": (412, 800, 2, 64, 9, 5, 900),              # 128 policies, a multiple of 64
        "rows1-one-resample": (413, 700, 3, 70, 6, 1, 1023),
        "rows2": (414, 1000, 3, 70, 17, 6, 1023),           # 210 policies: groups straddle rows
        "rows2-L33": (415, 600, 1, 130, 33, 4, 500),        # two load tiles
    }


def _tie_heavy(wl, cap):
    """Clip the waits below ``cap`` so that every timer whose deadline lies
    above the largest wait ties exactly with host-retain."""
    wl.wait_s = np.minimum(wl.wait_s, cap)
    return wl


def _check_fused(kvr, oracle_mod, wl, rows_vs_oracle):
    import torch
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    w, T, idx = _dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32()), _dev(wl.idx, _i32())
    lp = _lib_prices(kvr, wl)
    best, bc, cost = kvr.kvr_bootstrap(w, T, idx, lp, g, want_cost=True)
    nb, nbc = kvr.kvr_bootstrap(w, T, idx, lp, g)          # no cost tensor: same picks
    assert torch.equal(best, nb) and torch.equal(bc, nbc)
    # the selection rule applied to the GPU's own costs, on the host and by
    # kvr_select_policy: identical picks, best cost bit-equal to the pick's cost
    sel_b, sel_bc, _ = kvr.kvr_select_policy(cost, g.last_inf)
    assert torch.equal(best, sel_b)
    assert torch.equal(bc, sel_bc)
    c = _np(cost)
    hb, hbc, _ = oracle_mod.select(c, wl.t2)
    assert np.array_equal(_np(best), hb)
    assert np.array_equal(_np(bc), hbc)
    # exact ties were really exercised: count (resample, load) pairs whose
    # minimum is shared by several policies
    flat = c.reshape(c.shape[0], c.shape[1], -1)
    tied = int(((flat == flat.min(axis=2, keepdims=True)).sum(axis=2) > 1).sum())
    pr = oracle_mod.workload_prices(wl)
    for r in rows_vs_oracle:
        ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                   idx_row=wl.idx[r])
        assert_costs(c[r], ref)
        assert_selection(ref, _np(best)[r], oracle_mod.select(ref, wl.t2)[0])
    return tied


@pytest.mark.parametrize("name", sorted(_fused_plan_cases()))
def test_fused_argmin_tie_rule(kvr, oracle_mod, name):
    seed, n, k1, k2, L, R, m = _fused_plan_cases()[name]
    wl = _tie_heavy(workloads.random_case(seed, n, k1, k2, L, resamples=R, m=m, ties=True), 900.0)
    tied = _check_fused(kvr, oracle_mod, wl, rows_vs_oracle=range(R))
    print(f"[ties] {name}: {tied} (resample, load) minima shared by several policies")
    assert tied > 0


def _lane_layout_cases():
    # (seed, n, K1, K2, L, R, m): loads L <= 16 take tiles of 16, 8 or 4 loads
    return {
        "lt16-straddle": (420, 1000, 1, 257, 12, 5, 1000),   # groups straddle resamples
        "lt8-straddle": (417, 900, 3, 300, 7, 4, 1000),      # and t1 rows
        "lt4-straddle": (418, 800, 5, 256, 3, 3, 900),
        "lt4-rows": (419, 700, 2, 250, 4, 2, 1023),          # 500 policies per resample
    }


@pytest.mark.parametrize("split", [False, True], ids=["fused", "split"])
@pytest.mark.parametrize("name", sorted(_lane_layout_cases()))
def test_lane_layouts(kvr, oracle_mod, name, split):
    """Tiles of fewer than 32 loads with the selection fused into the grid
    kernel (one split) or over split partials (20,000 draws per resample):
    every cost against the oracle's double loop, the picks against the
    selection rule on the GPU's own costs, exactly."""
    seed, n, k1, k2, L, R, m = _lane_layout_cases()[name]
    if split:
        m = 20000
    wl = _tie_heavy(workloads.random_case(seed, n, k1, k2, L, resamples=R, m=m, ties=True), 900.0)
    tied = _check_fused(kvr, oracle_mod, wl, rows_vs_oracle=range(R))
    print(f"[ties] {name} {'split' if split else 'fused'}: {tied} shared minima")


@pytest.mark.parametrize("shape", [(421, 300000, 2, 256, 4), (422, 280000, 1, 257, 16),
                                   (423, 270000, 3, 300, 7)],
                         ids=["lt4", "lt16", "lt8"])
def test_lane_layouts_cost_grid(kvr, oracle_mod, shape):
    """kvr_cost_grid BRUTE on samples above the small-sample path (one
    resample, split partials) with tiles of 4, 16 and 8 loads: every cost
    against the oracle's double loop, and the selection."""
    seed, n, k1, k2, L = shape
    wl = workloads.random_case(seed, n, k1, k2, L, ties=True)
    cost, _, g = __import__("tests.test_gpu_parity", fromlist=["run_grid"]).run_grid(kvr, wl, "brute")
    pr = oracle_mod.workload_prices(wl)
    ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam)
    assert_costs(cost, ref)
    rb, _, _ = oracle_mod.select(ref, wl.t2)
    hb, _, _ = oracle_mod.select(cost, wl.t2)
    assert_selection(ref, hb, rb)


def test_fused_argmin_32k_waves(kvr, oracle_mod):
    """1,024 resamples x 514 policies x 128 loads: 32,896 base waves, so the
    selection is fused whatever the resample length (2,000 draws here)."""
    wl = _tie_heavy(workloads.random_case(416, 5000, 2, 257, 128, resamples=1024, m=2000,
                                          ties=True), 2000.0)
    tied = _check_fused(kvr, oracle_mod, wl, rows_vs_oracle=[0, 513, 1023])
    print(f"[ties] 32k waves: {tied} (resample, load) minima shared by several policies")
    assert tied > 0


def test_twotier_full_cost_tensors(kvr, oracle_mod):
    """The bench's two-tier launch (4,096 rows of 65,536 draws, 64 x 257
    policies, 32 loads) with the cost tensor kept: rows 0, 1,024, 2,048, 3,072
    and 4,095 element by element against the double loop (526,336 costs each),
    their selections, the selection rule on the GPU's own costs, and every
    row's picks equal to those of the launch without the tensor."""
    import torch
    wl = workloads.make("twotier-4096x64k")
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    w, T, idx = _dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32()), _dev(wl.idx, _i32())
    lp = _lib_prices(kvr, wl)
    nb, nbc = kvr.kvr_bootstrap(w, T, idx, lp, g)
    best, bc, cost = kvr.kvr_bootstrap(w, T, idx, lp, g, want_cost=True)
    assert torch.equal(best, nb) and torch.equal(bc, nbc)
    sel_b, sel_bc, _ = kvr.kvr_select_policy(cost, g.last_inf)
    assert torch.equal(best, sel_b) and torch.equal(bc, sel_bc)
    rows = [0, 1024, 2048, 3072, 4095]
    host = {r: _np(cost[r]) for r in rows}
    del cost, sel_b, sel_bc
    torch.cuda.empty_cache()
    pr = oracle_mod.workload_prices(wl)
    for r in rows:
        ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                   idx_row=wl.idx[r])
        assert ref.shape == (32, 64, 257)
        assert_costs(host[r], ref)
        hb, hbc, _ = oracle_mod.select(host[r], wl.t2)
        assert np.array_equal(_np(best)[r], hb) and np.array_equal(_np(bc)[r], hbc)
        rb, rbc, _ = oracle_mod.select(ref, wl.t2)
        n = assert_selection(ref, _np(best)[r], rb)
        assert_costs(_np(bc)[r], rbc)
        print(f"[twotier] row {r}: max rel err {H.rel_err(host[r], ref).max():.2e}, "
              f"{n} near-tie picks, smallest runner-up gap {H.min_runner_up_gap(ref):.2e}")


def test_tall_grid_many_t1_timers(kvr, oracle_mod):
    """2^20 GPU-tier timers x {300 s, inf}: the deadline count behind the
    recompute share searches along the short axis (two columns), so the call
    stays short; BRUTE, SORTED and a two-row bootstrap against the double loop."""
    import time
    import torch
    wl = workloads.random_case(421, 500, 1, 2, 1, resamples=2, ties=True)
    wl.t1 = np.concatenate([[0.0], np.geomspace(1e-3, 5000.0, (1 << 20) - 1)])
    assert np.all(np.diff(wl.t1) > 0)
    wl.t2 = np.array([300.0, np.inf])
    wl.lam = np.array([0.9])
    pr = oracle_mod.workload_prices(wl)
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    lp = _lib_prices(kvr, wl)
    w, T = _dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32())
    ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam)
    rb = oracle_mod.select(ref, wl.t2)[0]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    brute = kvr.kvr_cost_grid(w, T, lp, g, method=kvr.KVR_BRUTE)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    sorted_cost = kvr.kvr_cost_grid(w, T, lp, g, method=kvr.KVR_SORTED)
    for c in (brute, sorted_cost):
        assert_costs(_np(c), ref)
        assert_selection(ref, _np(kvr.kvr_select_policy(c, g.last_inf)[0]), rb)
    best, bc = kvr.kvr_bootstrap(w, T, _dev(wl.idx, _i32()), lp, g)
    for r in range(2):
        rr = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                  idx_row=wl.idx[r])
        rsel, rbc, _ = oracle_mod.select(rr, wl.t2)
        assert_selection(rr, _np(best)[r], rsel)
        assert_costs(_np(bc)[r], rbc)
    print(f"[tall] 2^21 policies, 500 waits: brute call {elapsed * 1e3:.1f} ms")
    assert elapsed < 5.0
