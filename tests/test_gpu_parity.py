"""GPU parity: the HIP library (through its C ABI) against the CPU oracle.

Bar: selected policy indices and sort order bit-exact; fp64 costs within
1e-9 relative.  Where two policies are within rounding of each other in the
oracle (a gap below 1e-11 relative, far below any real difference in these
workloads) either pick is accepted and the case is counted and printed.
"""
import math

import numpy as np
import pytest

import workloads
from tests import helpers as H

pytestmark = pytest.mark.gpu

RTOL = 1e-9          # fp64 cost tolerance
TIE_RTOL = 1e-11     # rounding-level near tie between two policies


@pytest.fixture(scope="module")
def kvr():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2608_30830_amd as k
    k.load_library()
    return k


def _dev(x, dtype):
    import torch
    return torch.as_tensor(np.ascontiguousarray(x)).to(device="cuda", dtype=dtype)


def _lib_prices(kvr, wl):
    pf = wl.platform
    return kvr.kvr_prices_from_platform(wl.kv_bytes_per_token, pf["hbm_usable_bytes"],
                                        pf["host_link_bytes_per_s"], pf["prefill_tokens_per_s"],
                                        pf["n_gpu"], pf["host_slots_c2"], pf["w_ref_s"])


def _np(t):
    return t.detach().cpu().numpy()


def assert_costs(gpu, ref, rtol=RTOL):
    gpu, ref = np.asarray(gpu), np.asarray(ref)
    assert gpu.shape == ref.shape
    err = H.rel_err(gpu, ref)
    worst = np.unravel_index(np.argmax(err), err.shape) if err.size else None
    assert err.max() <= rtol, f"max rel err {err.max():.3e} at {worst}: {gpu[worst]!r} vs {ref[worst]!r}"


def assert_selection(ref_cost, gpu_best, ref_best):
    """Identical indices, except rounding-level near ties (reported)."""
    n = H.near_tie_ok(ref_cost, gpu_best, ref_best, TIE_RTOL)
    if n:
        print(f"[near-tie] {n} selections differ within {TIE_RTOL:g} relative")
    return n


def run_grid(kvr, wl, method):
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    w, T = _dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32())
    if method == "sorted":
        cost, perm = kvr.kvr_cost_grid(w, T, _lib_prices(kvr, wl), g, method=kvr.KVR_SORTED,
                                       want_perm=True)
        return _np(cost), _np(perm), g
    cost = kvr.kvr_cost_grid(w, T, _lib_prices(kvr, wl), g, method=kvr.KVR_BRUTE)
    return _np(cost), None, g


def _f64():
    import torch
    return torch.float64


def _i32():
    import torch
    return torch.int32


RANDOM_CASES = [  # seed, n, K1, K2, L, ties  (ragged n, K2 below/at/above one wave)
    (101, 1, 1, 3, 1, False),
    (102, 7, 2, 5, 3, True),
    (103, 129, 1, 63, 5, True),
    (104, 1000, 3, 64, 17, True),
    (105, 4097, 2, 65, 33, True),
    (106, 3001, 1, 130, 40, False),
    (107, 2500, 4, 70, 9, True),
    (108, 300, 5, 2, 4, True),
    # eight t1 rows and ~4,000 finite deadlines over 16 pre-pass blocks: the
    # largest grid of the two-launch path for one sample
    (109, 16000, 8, 500, 5, True),
]


@pytest.mark.parametrize("case", RANDOM_CASES, ids=[f"seed{c[0]}" for c in RANDOM_CASES])
@pytest.mark.parametrize("method", ["brute", "sorted"])
def test_cost_grid_random(kvr, oracle_mod, case, method):
    seed, n, k1, k2, L, ties = case
    wl = workloads.random_case(seed, n, k1, k2, L, ties=ties)
    cost, perm, g = run_grid(kvr, wl, method)
    pr = oracle_mod.workload_prices(wl)
    ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam)
    assert_costs(cost, ref)
    if perm is not None:
        assert np.array_equal(perm, oracle_mod.stable_order(wl.wait_s))
    import torch
    best, bc, br = kvr.kvr_select_policy(torch.as_tensor(cost).cuda(), g.last_inf)
    rb, rbc, rbr = oracle_mod.select(ref, wl.t2)
    assert_selection(ref, _np(best), rb)
    assert_costs(_np(bc), rbc)
    if np.array_equal(_np(best), rb):
        assert np.array_equal(_np(br), rbr)


@pytest.mark.parametrize("name", ["tiny-exp-1k", "mix-64k"])
@pytest.mark.parametrize("method", ["brute", "sorted"])
def test_cost_grid_workloads(kvr, oracle_mod, name, method):
    """Full 1,000- and 65,536-wait workloads against the full oracle grid."""
    wl = workloads.make(name)
    cost, perm, g = run_grid(kvr, wl, method)
    pr = oracle_mod.workload_prices(wl)
    ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam)
    assert_costs(cost, ref)
    if perm is not None:
        assert np.array_equal(perm, oracle_mod.stable_order(wl.wait_s))
    import torch
    best, _, br = kvr.kvr_select_policy(torch.as_tensor(cost).cuda(), g.last_inf)
    rb, _, rbr = oracle_mod.select(ref, wl.t2)
    assert assert_selection(ref, _np(best), rb) == 0
    print(f"[gap] {name}/{method}: smallest best-vs-runner-up gap {H.min_runner_up_gap(ref):.3e}")


def test_tiny_workload_selects_as_the_memoryless_invariant_says(kvr):
    """The 1,000 exponential waits: retain at 0.25/s, the shortest timer above
    the threshold load (the same pin the oracle carries)."""
    wl = workloads.make("tiny-exp-1k")
    cost, _, g = run_grid(kvr, wl, "brute")
    import torch
    best, _, br = kvr.kvr_select_policy(torch.as_tensor(cost).cuda(), g.last_inf)
    assert list(_np(best)) == [64, 0, 0, 0]
    assert list(_np(br)) == [kvr.KVR_RETAIN, kvr.KVR_EXPIRE, kvr.KVR_EXPIRE, kvr.KVR_EXPIRE]


def test_weibull_1m_sorted_brute_and_sampled_oracle(kvr, oracle_mod):
    """1,048,576 waits, 1,025 timers, 64 loads: BRUTE and SORTED against the
    oracle's closed form on the full grid, the double loop on sampled timer
    columns, and the stable order bit for bit."""
    wl = workloads.make("weibull-1m")
    pr = oracle_mod.workload_prices(wl)
    cb, _, g = run_grid(kvr, wl, "brute")
    cs, perm, _ = run_grid(kvr, wl, "sorted")
    ref_perm = oracle_mod.stable_order(wl.wait_s)
    assert np.array_equal(perm, ref_perm)
    closed = oracle_mod.closed_form_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                         perm=ref_perm)
    assert_costs(cb, closed)
    assert_costs(cs, closed)
    cols = np.unique(np.concatenate([np.arange(0, wl.t2.size, 97), [wl.t2.size - 2,
                                                                      wl.t2.size - 1]]))
    ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2[cols], wl.lam)
    assert_costs(cb[:, :, cols], ref)
    assert_costs(cs[:, :, cols], ref)
    import torch
    b1 = _np(kvr.kvr_select_policy(torch.as_tensor(cb).cuda(), g.last_inf)[0])
    b2 = _np(kvr.kvr_select_policy(torch.as_tensor(cs).cuda(), g.last_inf)[0])
    rb = oracle_mod.select(closed, wl.t2)[0]
    assert_selection(closed, b1, rb)
    assert_selection(closed, b2, rb)


def test_max_size_2p24_waits(kvr, oracle_mod):
    """2^24 waits, sixteen times the largest workload (the sorted path's
    scaling sample): the stable order bit for bit, and BRUTE and SORTED against
    the oracle's closed form on the whole grid, with every selection."""
    wl = workloads.sort_scale_case(24)
    pr = oracle_mod.workload_prices(wl)
    cb, _, g = run_grid(kvr, wl, "brute")
    cs, perm, _ = run_grid(kvr, wl, "sorted")
    ref_perm = oracle_mod.stable_order(wl.wait_s)
    assert np.array_equal(perm, ref_perm)
    closed = oracle_mod.closed_form_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                         perm=ref_perm)
    assert_costs(cb, closed)
    assert_costs(cs, closed)
    import torch
    rb = oracle_mod.select(closed, wl.t2)[0]
    for c in (cb, cs):
        assert_selection(closed, _np(kvr.kvr_select_policy(torch.as_tensor(c).cuda(),
                                                           g.last_inf)[0]), rb)


@pytest.mark.parametrize("n", [(1 << 22) - 1, (1 << 22) + 1001, (1 << 23) + 4095],
                         ids=["2p22-1-keys", "2p22+1001-kpt8", "2p23+4095-kpt16"])
def test_sorted_digit_byte_passes(kvr, oracle_mod, n):
    """From 2^22 waits each digit pass counts the digit bytes that the
    previous scatter wrote instead of reading the keys (one below that, the
    keys): ragged samples at 8 and 16 keys per thread, with duplicated waits
    and both signed zeros; the stable order bit for bit, and the costs with
    and without a requested order against the oracle's closed form."""
    wl = workloads.random_case(300 + n % 97, n, 2, 40, 4, ties=True)
    rng = np.random.default_rng(n)
    wl.wait_s[rng.integers(0, n, n // 64)] = -0.0   # sorts as +0.0, in input order
    pr = oracle_mod.workload_prices(wl)
    cs, perm, g = run_grid(kvr, wl, "sorted")
    ref_perm = oracle_mod.stable_order(wl.wait_s)
    assert np.array_equal(perm, ref_perm)
    closed = oracle_mod.closed_form_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                         perm=ref_perm)
    assert_costs(cs, closed)
    cost = kvr.kvr_cost_grid(_dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32()),
                             _lib_prices(kvr, wl), g, method=kvr.KVR_SORTED)
    assert_costs(_np(cost), closed)


@pytest.mark.parametrize("case", [(201, 500, 2, 70, 5, 3, None), (202, 1300, 1, 65, 16, 4, 777),
                                  (203, 64, 3, 9, 3, 5, 200), (204, 2000, 2, 128, 33, 2, None),
                                  # few resamples, many draws: several recompute-share blocks
                                  # per resample add into one row
                                  (205, 5000, 2, 70, 6, 2, 20000)])
def test_bootstrap_random(kvr, oracle_mod, case):
    seed, n, k1, k2, L, R, m = case
    wl = workloads.random_case(seed, n, k1, k2, L, resamples=R, m=m, ties=True)
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    best, bc, cost = kvr.kvr_bootstrap(_dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32()),
                                       _dev(wl.idx, _i32()), _lib_prices(kvr, wl), g,
                                       want_cost=True)
    pr = oracle_mod.workload_prices(wl)
    for r in range(R):
        ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                   idx_row=wl.idx[r])
        assert_costs(_np(cost)[r], ref)
        rb, rbc, _ = oracle_mod.select(ref, wl.t2)
        assert_selection(ref, _np(best)[r], rb)
        assert_costs(_np(bc)[r], rbc)
    # without the cost tensor the selection is the same
    best2, bc2 = kvr.kvr_bootstrap(_dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32()),
                                   _dev(wl.idx, _i32()), _lib_prices(kvr, wl), g)
    assert np.array_equal(_np(best2), _np(best))
    assert_costs(_np(bc2), _np(bc), rtol=1e-15)


@pytest.mark.parametrize("seed,n,k1,k2,L", [(211, 3000, 3, 70, 5), (212, 700, 2, 9, 33)])
def test_offload_charge_every_grid_method(kvr, oracle_mod, seed, n, k1, k2, L):
    """The optional charge for the copy at offload (T * b2 per request with
    w > t1, the link's per-token time) through BRUTE, SORTED, the bootstrap
    and the factored bootstrap, against the oracle's double loop with the
    same charge."""
    wl = workloads.random_case(seed, n, k1, k2, L, resamples=3, ties=True)
    pf = wl.platform
    args = (wl.kv_bytes_per_token, pf["hbm_usable_bytes"], pf["host_link_bytes_per_s"],
            pf["prefill_tokens_per_s"], pf["n_gpu"], pf["host_slots_c2"], pf["w_ref_s"])
    lp = kvr.kvr_prices_from_platform(*args, charge_offload=True)
    pr = oracle_mod.prices_from_platform(*args, charge_offload=True)
    assert lp.offload_per_token == pr.boff > 0.0
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    w, T = _dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32())
    ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam)
    for method in (kvr.KVR_BRUTE, kvr.KVR_SORTED):
        cost = kvr.kvr_cost_grid(w, T, lp, g, method=method)
        assert_costs(_np(cost), ref)
        assert_selection(ref, _np(kvr.kvr_select_policy(cost, g.last_inf)[0]),
                         oracle_mod.select(ref, wl.t2)[0])
    idx = _dev(wl.idx, _i32())
    for factored in (False, True):
        best, bc, cost = kvr.kvr_bootstrap(w, T, idx, lp, g, want_cost=True, factored=factored)
        for r in range(3):
            rr = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                      idx_row=wl.idx[r])
            assert_costs(_np(cost)[r], rr)
            rb, rbc, _ = oracle_mod.select(rr, wl.t2)
            assert_selection(rr, _np(best)[r], rb)
            assert_costs(_np(bc)[r], rbc)


def _boot_full(kvr, oracle_mod, name, sample_rows):
    wl = workloads.make(name)
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    best, bc = kvr.kvr_bootstrap(_dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32()),
                                 _dev(wl.idx, _i32()), _lib_prices(kvr, wl), g)
    best, bc = _np(best), _np(bc)
    pr = oracle_mod.workload_prices(wl)
    # every row: the closed form's selection and best cost
    cb, cbc = oracle_mod.closed_form_bootstrap(wl.wait_s, wl.ctx_tokens, wl.idx, pr, wl.t1,
                                               wl.t2, wl.lam)
    assert_costs(bc, cbc)
    differ = np.argwhere(best != cb)
    rows = {}
    for r, l in differ:
        # must be a rounding-level tie of the closed form itself: the reference
        # cost of the GPU's pick is within TIE_RTOL of the reference best
        if r not in rows:
            rows[r] = oracle_mod.closed_form_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2,
                                                  wl.lam, idx_row=wl.idx[r])
        ref_l = rows[r][l].ravel()
        assert ref_l[best[r, l]] - ref_l.min() <= TIE_RTOL * abs(ref_l.min()), (r, l)
        assert abs(bc[r, l] - cbc[r, l]) <= TIE_RTOL * abs(cbc[r, l]) + RTOL * abs(cbc[r, l])
    print(f"[boot] {name}: {len(differ)} of {best.size} selections differ from the closed form")
    # sampled rows: the double loop, element by element
    for r in sample_rows:
        ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam,
                                   idx_row=wl.idx[r])
        rb, rbc, _ = oracle_mod.select(ref, wl.t2)
        assert_selection(ref[None], best[r][None], rb[None])
        assert_costs(bc[r], rbc)
    return wl


def test_bootstrap_1024_full(kvr, oracle_mod):
    _boot_full(kvr, oracle_mod, "boot-1024x64k", sample_rows=[0, 511, 1023])


def test_bootstrap_twotier_4096_full(kvr, oracle_mod):
    """The two-tier workload at full size, in the launch configuration the
    benchmark times: all 4,096 rows against the closed form, two rows against
    the double loop."""
    _boot_full(kvr, oracle_mod, "twotier-4096x64k", sample_rows=[0, 4095])


@pytest.mark.parametrize("k1", [2, 9])
def test_identity_rows_equal_cost_grid(kvr, k1):
    """A bootstrap row drawing every sample once in order is the plain grid:
    bit for bit where both calls run the same kernels in the same order (nine
    GPU-tier timers), within 1e-12 where the plain grid of one small sample
    adds its splits in blocks (two timers, the two-launch path)."""
    wl = workloads.random_case(301, 5000, k1, 66, 6)
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    idx = np.tile(np.arange(wl.n, dtype=np.int32), (3, 1))
    best, bc, cost = kvr.kvr_bootstrap(_dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32()),
                                       _dev(idx, _i32()), _lib_prices(kvr, wl), g, want_cost=True)
    plain, _, _ = run_grid(kvr, wl, "brute")
    for r in range(3):
        if k1 > 8:
            assert np.array_equal(_np(cost)[r], plain)
        else:
            assert_costs(_np(cost)[r], plain, rtol=1e-12)


def test_deterministic(kvr):
    wl = workloads.random_case(302, 30000, 3, 100, 20, resamples=4)
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    args = (_dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32()), _dev(wl.idx, _i32()),
            _lib_prices(kvr, wl), g)
    a = kvr.kvr_bootstrap(*args, want_cost=True)
    b = kvr.kvr_bootstrap(*args, want_cost=True)
    for x, y in zip(a, b):
        assert np.array_equal(_np(x), _np(y))
    c1, _, _ = run_grid(kvr, wl, "sorted")
    c2, _, _ = run_grid(kvr, wl, "sorted")
    assert np.array_equal(c1, c2)


def test_structural_ties_exact(kvr, oracle_mod):
    """Waits all below the largest timers: every such timer ties with
    host-retain exactly, and the tie goes to host-retain (larger index)."""
    rng = np.random.Generator(np.random.PCG64(9))
    n = 3000
    w = rng.uniform(0, 500.0, n)
    T = rng.integers(1, 30000, n).astype(np.int32)
    t1 = np.array([0.0, 20.0])
    t2 = np.concatenate([np.geomspace(1, 2000, 70), [np.inf]])
    lam = np.array([0.1, 0.3, 0.9, 2.0])
    wl = workloads.Workload("ties", w, T, t1, t2, lam, float(workloads.KV_128K))
    cost, _, g = run_grid(kvr, wl, "brute")
    cs, _, _ = run_grid(kvr, wl, "sorted")
    tied = t2[:-1] + 20.0 >= w.max()
    for c in (cost, cs):
        for a in range(2):
            for k in np.nonzero(tied)[0]:
                assert np.array_equal(c[:, a, k], c[:, a, -1])
    pr = oracle_mod.workload_prices(wl)
    ref = oracle_mod.cost_grid(w, T, pr, t1, t2, lam)
    import torch
    for c in (cost, cs):
        best = _np(kvr.kvr_select_policy(torch.as_tensor(c).cuda(), 1)[0])
        assert np.array_equal(best, oracle_mod.select(ref, t2)[0])


def test_domain_errors_are_reported(kvr):
    """Bad samples or indices set the status word; nothing faults."""
    import torch
    wl = workloads.random_case(303, 2000, 1, 65, 3, resamples=2)
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    pr = _lib_prices(kvr, wl)
    for bad in ("nan", "neg", "inf"):
        w = wl.wait_s.copy()
        w[17] = {"nan": np.nan, "neg": -3.0, "inf": np.inf}[bad]
        for method in (kvr.KVR_BRUTE, kvr.KVR_SORTED):
            with pytest.raises(kvr.KvrError) as ei:
                kvr.kvr_cost_grid(_dev(w, _f64()), _dev(wl.ctx_tokens, _i32()), pr, g,
                                  method=method)
            assert ei.value.code == kvr.KVR_E_DOMAIN
    T = wl.ctx_tokens.copy()
    T[3] = 0
    with pytest.raises(kvr.KvrError) as ei:
        kvr.kvr_cost_grid(_dev(wl.wait_s, _f64()), _dev(T, _i32()), pr, g)
    assert ei.value.code == kvr.KVR_E_DOMAIN
    for badidx in (-1, wl.n):
        idx = wl.idx.copy()
        idx[1, 5] = badidx
        with pytest.raises(kvr.KvrError) as ei:
            kvr.kvr_bootstrap(_dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32()),
                              _dev(idx, _i32()), pr, g)
        assert ei.value.code == kvr.KVR_E_DOMAIN
    # a clean call afterwards on a fresh workspace reports OK
    kvr.kvr_cost_grid(_dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32()), pr, g)
    torch.cuda.synchronize()


def test_binding_rejects_mismatched_arguments(kvr):
    """The binding checks what the C ABI cannot see (tensor shapes, dtypes,
    devices) and raises before anything is launched."""
    import torch
    wl = workloads.random_case(304, 500, 1, 9, 3, resamples=2)
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    pr = _lib_prices(kvr, wl)
    w, T = _dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32())
    with pytest.raises(ValueError):
        kvr.kvr_cost_grid(w, T[:-1], pr, g)                                  # short contexts
    with pytest.raises(ValueError):
        kvr.kvr_cost_grid(w, T, pr, g, out=torch.empty((3, 1, 8), dtype=torch.float64,
                                                        device="cuda"))      # small output
    with pytest.raises(ValueError):
        kvr.kvr_cost_grid(w, T, pr, g, out=torch.empty((3, 1, 9), dtype=torch.float32,
                                                        device="cuda"))      # wrong dtype
    with pytest.raises(ValueError):
        kvr.kvr_cost_grid(w, T, pr, g, workspace=torch.empty(1 << 20, dtype=torch.float64,
                                                              device="cuda"))
    with pytest.raises(ValueError):
        kvr.kvr_cost_grid(w.cpu(), T, pr, g)                                 # host tensor
    with pytest.raises(ValueError):
        kvr.kvr_bootstrap(w, T[:-1], _dev(wl.idx, _i32()), pr, g)
    arr = torch.cumsum(torch.ones((2, 50), dtype=torch.float64, device="cuda"), 1)
    with pytest.raises(ValueError):
        kvr.kvr_capacity_replay(arr, arr.clone(), pr, [60.0],
                                ctx_tokens=torch.ones((2, 49), dtype=torch.int32, device="cuda"))
    cost = kvr.kvr_cost_grid(w, T, pr, g)                                    # a valid call
    assert tuple(cost.shape) == (3, 1, 9)


PROFILED_CALLS = ["bootstrap", "bootstrap_factored", "cost_grid_brute", "cost_grid_sorted",
                  "capacity_replay", "controller_select"]


@pytest.mark.parametrize("entry", PROFILED_CALLS)
def test_profile_events_bracket_the_main_stage(kvr, entry):
    """kvr_set_profile_events: every entry point that documents it records the
    caller's two events around its main stage on the call's stream (fresh,
    never-recorded events, so a call that skips them fails the elapsed-time
    query)."""
    import ctypes
    import torch
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                        ctypes.c_void_p]
    hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
    evs = [ctypes.c_void_p(), ctypes.c_void_p()]
    for e in evs:
        assert hip.hipEventCreate(ctypes.byref(e)) == 0
    wl = workloads.random_case(304, 20000, 2, 80, 8, resamples=8)
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    w, T = _dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32())
    pr = _lib_prices(kvr, wl)
    if entry in ("capacity_replay", "controller_select"):
        rc = workloads.replay_case("mixture", 0.5, reps=2, n=1000, seed=5)
        arr, rw = _dev(rc.arrival_s, _f64()), _dev(rc.wait_s, _f64())
    calls = {
        "bootstrap": lambda: kvr.kvr_bootstrap(w, T, _dev(wl.idx, _i32()), pr, g),
        "bootstrap_factored": lambda: kvr.kvr_bootstrap(w, T, _dev(wl.idx, _i32()), pr, g,
                                                        factored=True),
        "cost_grid_brute": lambda: kvr.kvr_cost_grid(w, T, pr, g, kvr.KVR_BRUTE),
        "cost_grid_sorted": lambda: kvr.kvr_cost_grid(w, T, pr, g, kvr.KVR_SORTED),
        "capacity_replay": lambda: kvr.kvr_capacity_replay(arr, rw, pr, [60.0, float("inf")]),
        "controller_select": lambda: kvr.kvr_controller_select(arr, rw, pr, 0.5),
    }
    kvr.kvr_set_profile_events(evs[0].value, evs[1].value)
    try:
        calls[entry]()
    finally:
        kvr.kvr_set_profile_events(None, None)
    torch.cuda.synchronize()
    ms = ctypes.c_float()
    assert hip.hipEventElapsedTime(ctypes.byref(ms), evs[0], evs[1]) == 0
    assert ms.value > 0.0
    for e in evs:
        hip.hipEventDestroy(e)
    with pytest.raises(kvr.KvrError):
        kvr.kvr_set_profile_events(evs[0].value, None)


DEGENERATE = {
    # every wait zero: every policy costs 0 (ties everywhere, largest index wins)
    "all-zero": (np.zeros(300), np.full(300, 7, np.int32), np.array([0.0, 5.0]),
                 np.array([1.0, 2.0, np.inf]), np.array([0.1, 0.9])),
    # every wait sits exactly on a deadline t1 + t2
    "on-deadline": (np.full(200, 30.0 + 45.0), np.arange(1, 201, dtype=np.int32),
                    np.array([0.0, 30.0]), np.array([10.0, 45.0, 80.0, np.inf]),
                    np.array([0.2, 0.5, 3.0])),
    # host-retain only
    "retain-only": (np.linspace(0.0, 5000.0, 777), np.full(777, 4096, np.int32),
                    np.array([0.0]), np.array([np.inf]), np.array([0.05, 0.3, 1.0])),
    # every load at or below lambda_crit: no congestion price
    "uncongested": (np.geomspace(1.0, 20000.0, 1500), np.full(1500, 1000, np.int32),
                    np.array([0.0, 2.0, 9.0]), np.concatenate([np.geomspace(3, 9000, 70), [np.inf]]),
                    np.array([0.0, 0.1, 425.0 / 1800.0])),
    # one sample, one timer pair, one load
    "single": (np.array([123.0]), np.array([5], np.int32), np.array([0.0]), np.array([100.0]),
               np.array([0.7])),
    # deadlines repeated across t1 rows (10+20 = 20+10 = ...), waits on them and one ulp above
    "dup-deadlines": (np.concatenate([np.repeat([10.0, 20.0, 30.0, 40.0, 50.0], 40),
                                      np.nextafter([10.0, 20.0, 30.0, 40.0, 50.0], np.inf),
                                      np.geomspace(1.0, 90.0, 395)]),
                      np.arange(1, 601, dtype=np.int32), np.array([0.0, 10.0, 20.0]),
                      np.array([10.0, 20.0, 30.0, np.inf]), np.array([0.1, 0.5, 2.0])),
    # t1 + t2 overflows to +inf for a finite t2: that deadline is never reached
    "overflow": (np.concatenate([np.geomspace(1.0, 1e306, 300), [0.0, 1e300]]),
                 np.full(302, 3, np.int32), np.array([0.0, 1e308]),
                 np.array([1e300, 1e308, np.inf]), np.array([0.05, 0.2])),
    # many t1 rows, one host timer (group straddles rows every lane)
    "k2-one": (np.geomspace(0.5, 9000.0, 640), np.full(640, 33, np.int32),
               np.geomspace(0.1, 3000.0, 150), np.array([60.0]), np.array([0.4, 0.8])),
}


@pytest.mark.parametrize("name", sorted(DEGENERATE))
@pytest.mark.parametrize("method", ["brute", "sorted"])
def test_degenerate_inputs(kvr, oracle_mod, name, method):
    w, T, t1, t2, lam = DEGENERATE[name]
    wl = workloads.Workload(name, w.astype(np.float64), T, t1, t2, lam, float(workloads.KV_128K))
    cost, perm, g = run_grid(kvr, wl, method)
    pr = oracle_mod.workload_prices(wl)
    ref = oracle_mod.cost_grid(wl.wait_s, wl.ctx_tokens, pr, wl.t1, wl.t2, wl.lam)
    if np.all(ref == 0):
        assert np.all(cost == 0)
    else:
        assert_costs(cost, ref)
    if perm is not None:
        assert np.array_equal(perm, oracle_mod.stable_order(wl.wait_s))
    import torch
    best, _, br = kvr.kvr_select_policy(torch.as_tensor(cost).cuda(), g.last_inf)
    rb, _, rbr = oracle_mod.select(ref, wl.t2)
    assert np.array_equal(_np(best), rb)
    assert np.array_equal(_np(br), rbr)


def test_batched_select_matches_fused_selection(kvr):
    """kvr_select_policy over a [R, L, K1, K2] cost tensor picks what the
    bootstrap's fused per-wave selection picked."""
    wl = workloads.random_case(305, 6000, 3, 90, 12, resamples=6, ties=True)
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    best, bc, cost = kvr.kvr_bootstrap(_dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32()),
                                       _dev(wl.idx, _i32()), _lib_prices(kvr, wl), g,
                                       want_cost=True)
    b2, bc2, br2 = kvr.kvr_select_policy(cost, g.last_inf)
    assert np.array_equal(_np(best), _np(b2))
    assert np.array_equal(_np(bc), _np(bc2))
    assert tuple(b2.shape) == (6, wl.lam.size)
