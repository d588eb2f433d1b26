"""GPU parity of the multiplicity-count closed form (kvr_bootstrap_factored):
against the oracle's double loop on random bootstrap rows (costs within
1e-9 relative), against the oracle's closed-form selection on every row of
the bench bootstrap workloads, and against the brute-force kvr_bootstrap on
the same rows (selection identical up to rounding-level near ties: where two
picks differ, their best costs agree to rounding)."""
import numpy as np
import pytest

import workloads
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


def _factored(kvr, wl, want_cost=False, prices=None):
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    return kvr.kvr_bootstrap(_dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32()),
                             _dev(wl.idx, _i32()), prices or _lib_prices(kvr, wl), g,
                             want_cost=want_cost, factored=True)


@pytest.mark.parametrize("case", [(201, 500, 2, 70, 5, 3, None), (202, 1300, 1, 65, 16, 4, 777),
                                  (203, 64, 3, 9, 3, 5, 200), (204, 2000, 2, 128, 33, 2, None),
                                  (206, 40000, 1, 80, 40, 3, 30000)])
def test_factored_random(kvr, oracle_mod, case):
    seed, n, k1, k2, L, R, m = case
    wl = workloads.random_case(seed, n, k1, k2, L, resamples=R, m=m, ties=True)
    best, bc, cost = _factored(kvr, wl, want_cost=True)
    pr = oracle_mod.workload_prices(wl)
    for r in range(R):
        ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                   idx_row=wl.idx[r])
        assert_costs(_np(cost)[r], ref)
        rb, rbc, _ = oracle_mod.select(ref, wl.t2)
        assert_selection(ref, _np(best)[r], rb)
        assert_costs(_np(bc)[r], rbc)
    best2, bc2 = _factored(kvr, wl)
    assert np.array_equal(_np(best2), _np(best))
    assert np.array_equal(_np(bc2), _np(bc))


def _rows_agree(got, got_cost, want, want_cost, label, ref_row):
    """Where two selections differ, the two picks' best costs must agree to
    rounding, and under the oracle's closed form of that row (ref_row(r):
    cost[L, K1, K2]) both picks must lie within TIE_RTOL of the best (a near
    tie); returns how many selections differ."""
    differ = np.argwhere(got != want)
    rows = {}
    for r, l in differ:
        a, b = got_cost[r, l], want_cost[r, l]
        assert abs(a - b) <= (TIE_RTOL + RTOL) * abs(b), (label, r, l, a, b)
        if r not in rows:
            rows[r] = ref_row(r)
        ref_l = rows[r][l].ravel()
        lo = ref_l.min()
        for pick in (got[r, l], want[r, l]):
            assert ref_l[pick] - lo <= TIE_RTOL * abs(lo), (label, r, l, pick)
    print(f"[near-tie] {label}: {len(differ)} of {got.size} selections differ")
    return len(differ)


@pytest.mark.parametrize("name", ["boot-1024x64k", "twotier-4096x64k"])
def test_factored_bench_workloads(kvr, oracle_mod, name):
    wl = workloads.make(name)
    fb, fbc = _factored(kvr, wl)
    fb, fbc = _np(fb), _np(fbc)
    pr = oracle_mod.workload_prices(wl)
    cb, cbc = oracle_mod.closed_form_bootstrap(wl.wait_s, wl.ctx_tokens, wl.idx, pr, wl.t1,
                                               wl.t2, wl.lam)
    assert_costs(fbc, cbc)

    def ref_row(r):
        return oracle_mod.closed_form_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                           idx_row=wl.idx[r])
    _rows_agree(fb, fbc, cb, cbc, f"{name} factored vs oracle closed form", ref_row)
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    bb, bbc = kvr.kvr_bootstrap(_dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32()),
                                _dev(wl.idx, _i32()), _lib_prices(kvr, wl), g)
    assert_costs(fbc, _np(bbc))
    _rows_agree(fb, fbc, _np(bb), _np(bbc), f"{name} factored vs brute", ref_row)
    # sampled rows against the double loop, element by element
    for r in (0, wl.n_resamples - 1):
        ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                   idx_row=wl.idx[r])
        rb, rbc, _ = oracle_mod.select(ref, wl.t2)
        assert_selection(ref[None], fb[r][None], rb[None])
        assert_costs(fbc[r], rbc)


def test_factored_platforms(kvr, oracle_mod):
    wl = workloads.cross_platform_case()
    for name, (a1, b2, b3) in workloads.PLATFORM_PRICES.items():
        p = kvr.kvr_prices_from_platform(1.0, 1.0, 1.0, 1.0, 1.0, 425.0, 1800.0)
        p.a1_per_token, p.b2_per_token, p.b3_per_token = a1, b2, b3
        best, bc, cost = _factored(kvr, wl, want_cost=True, prices=p)
        pr = oracle_mod.Prices(a1, b2, b3)
        for r in range(3):
            ref = oracle_mod.closed_form_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                              idx_row=wl.idx[r])
            assert_costs(_np(cost)[r], ref)
            rb, _, _ = oracle_mod.select(ref, wl.t2)
            assert_selection(ref, _np(best)[r], rb)


def test_factored_domain_errors(kvr):
    wl = workloads.random_case(207, 300, 1, 70, 4, resamples=2, m=300)
    for what in ("idx", "nan"):
        w, idx = wl.wait_s.copy(), wl.idx.copy()
        if what == "idx":
            idx[1, 5] = wl.n
        else:
            w[17] = np.nan
        g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
        with pytest.raises(kvr.KvrError) as ei:
            kvr.kvr_bootstrap(_dev(w, _f64()), _dev(wl.ctx_tokens, _i32()), _dev(idx, _i32()),
                              _lib_prices(kvr, wl), g, factored=True)
        assert ei.value.code == kvr.KVR_E_DOMAIN


@pytest.mark.parametrize("n", [1000, 100000])
def test_factored_heavy_multiplicities(kvr, oracle_mod, n):
    """Rows that draw one base sample 15 or 16 times (the largest count a 4-bit
    multiplicity counter holds, and one more, in the lowest, a middle and the
    top field of an LDS word), 256, 65,535, 65,536 or 70,000 times, so that a
    narrow counter wraps (or just does not): the kernel must detect a wrap
    and recount the row with 32-bit counters.  With n = 1,000 the draws are
    counted by base sample; with n = 100,000 by sorted position, in two
    passes."""
    m = 70000
    wl = workloads.random_case(208, n, 1, 9, 3, resamples=10, m=m, ties=True)
    order = np.argsort(wl.wait_s, kind="stable")
    rng = np.random.Generator(np.random.PCG64(209))
    idx = rng.integers(0, n, size=(10, m), dtype=np.int32)
    pos = lambda k: int(order[k])                    # the sample at sorted position k
    idx[0, :] = pos(10)                               # 70,000 draws of one sample
    idx[1, :] = pos(11)
    idx[2, :65536] = pos(10)                          # exactly 65,536
    idx[3, :65536] = pos(11)
    idx[4, :65535] = pos(11)
    for row, (sample, times) in zip((5, 6, 7), ((8, 15), (12, 16), (15, 16))):
        idx[row][idx[row] == sample] = sample + 1     # exactly `times` draws of `sample`:
        idx[row, :times] = sample                     # 15 fit a 4-bit field (word 1, field 0),
                                                      # 16 wrap a middle and the top field
    idx[8, :256] = pos(13)
    wl.idx = idx                                      # row 9 stays random
    best, bc, cost = _factored(kvr, wl, want_cost=True)
    pr = oracle_mod.workload_prices(wl)
    for r in range(10):
        ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                   idx_row=idx[r])
        assert_costs(_np(cost)[r], ref)
        rb, rbc, _ = oracle_mod.select(ref, wl.t2)
        assert_selection(ref, _np(best)[r], rb)
        assert_costs(_np(bc)[r], rbc)


def test_factored_many_draws_integer_sums(kvr, oracle_mod):
    """More than 2^22 draws per resample: the prefix kernel carries the N sums
    in 64-bit integers (below that, in doubles, exact while m times a context
    size stays below 2^53); costs and selections against the oracle's double
    loop."""
    m = (1 << 22) + 7
    wl = workloads.random_case(210, 3000, 1, 9, 3, resamples=2, m=m, ties=True)
    best, bc, cost = _factored(kvr, wl, want_cost=True)
    pr = oracle_mod.workload_prices(wl)
    for r in range(2):
        ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                   idx_row=wl.idx[r])
        assert_costs(_np(cost)[r], ref)
        rb, rbc, _ = oracle_mod.select(ref, wl.t2)
        assert_selection(ref, _np(best)[r], rb)
        assert_costs(_np(bc)[r], rbc)


@pytest.mark.parametrize("name", sorted(__import__("tests.test_gpu_parity",
                                                   fromlist=["DEGENERATE"]).DEGENERATE))
def test_factored_degenerate_inputs(kvr, oracle_mod, name):
    """The grid's degenerate cases (every wait zero, waits on deadlines, retain
    only, no congestion, one sample, repeated deadlines, t1 + t2 overflowing to
    +inf, one host timer) through the factored method, with an identity row
    and a seeded row: costs and selections against the oracle."""
    from tests.test_gpu_parity import DEGENERATE
    w, T, t1, t2, lam = DEGENERATE[name]
    n = w.size
    rng = np.random.Generator(np.random.PCG64(300 + n))
    idx = np.stack([np.arange(n, dtype=np.int32), rng.integers(0, n, n, dtype=np.int32)])
    wl = workloads.Workload(name, w.astype(np.float64), T, t1, t2, lam,
                            float(workloads.KV_128K), idx=idx)
    best, bc, cost = _factored(kvr, wl, want_cost=True)
    pr = oracle_mod.workload_prices(wl)
    for r in range(2):
        ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                   idx_row=idx[r])
        assert_costs(_np(cost)[r], ref)
        rb, rbc, _ = oracle_mod.select(ref, wl.t2)
        assert_selection(ref, _np(best)[r], rb)
        assert_costs(_np(bc)[r], rbc)


def _tie_case(name, k1):
    rng = np.random.Generator(np.random.PCG64(700 + k1))
    if name == "all-zero":
        # every policy costs exactly 0
        w = np.zeros(3000)
        t2 = np.concatenate([np.geomspace(1.0, 1e5, 300), [np.inf]])
    else:
        # loads at or below lambda_crit (no holding price) and about three
        # deadlines per gap between waits: the policies of one t1 row whose
        # deadlines share a gap cost exactly the same
        w = np.geomspace(1.0, 1e4, 500)
        t2 = np.concatenate([np.geomspace(1.0, 1e5, 2000), [np.inf]])
    T = rng.integers(1, 5000, w.size).astype(np.int32)
    t1 = np.array([0.0, 5.0, 50.0, 400.0, 900.0, 3000.0, 7000.0])[:k1]
    lam = np.array([0.05, 0.1, 425.0 / 1800.0])
    idx = np.stack([np.arange(w.size, dtype=np.int32),
                    rng.integers(0, w.size, w.size, dtype=np.int32)])
    return workloads.Workload(name, w, T, t1, t2, lam, float(workloads.KV_128K), idx=idx)


@pytest.mark.parametrize("name", ["all-zero", "gap-ties"])
@pytest.mark.parametrize("k1", [1, 7])
def test_factored_exact_tie_rule(kvr, oracle_mod, name, k1):
    """Exact ties with one and with several t1 rows (all-zero waits: every
    policy ties; gap ties: the policies of a t1 row whose deadlines share a
    gap between waits tie below lambda_crit): every selection is the largest
    flat index among the policies whose cost equals the minimum, on the GPU's
    own cost tensor, and equals the oracle's."""
    wl = _tie_case(name, k1)
    best, bc, cost = _factored(kvr, wl, want_cost=True)
    best, bc, cost = _np(best), _np(bc), _np(cost)
    R, L = best.shape
    nties = 0
    for r in range(R):
        for l in range(L):
            c = cost[r, l].ravel()
            at_min = np.flatnonzero(c == c.min())
            nties += at_min.size > 1
            assert best[r, l] == at_min[-1], (r, l, best[r, l], at_min[-8:])
            assert bc[r, l] == c.min()
    assert nties >= R * L // 2, nties
    pr = oracle_mod.workload_prices(wl)
    for r in range(R):
        ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                   idx_row=wl.idx[r])
        assert_costs(cost[r], ref)
        rb, _, _ = oracle_mod.select(ref, wl.t2)
        assert np.array_equal(best[r], rb), (r, best[r], rb)
