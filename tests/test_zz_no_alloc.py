"""kvr_cost_grid_noalloc (the library's static device scratch as workspace)
against kvr_cost_grid (a caller-sized workspace), through the C ABI: two calls
in a row, the second with a smaller input, per method; a plan that has to take
fewer sample splits to fit the scratch; the status word; the size limit."""
import numpy as np
import pytest

import workloads
from tests.test_gpu_parity import (_dev, _f64, _i32, _lib_prices, _np, assert_costs,
                                   assert_selection)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kvr():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2608_30830_amd as k
    k.load_library()
    return k


def _both(kvr, wl, method):
    import torch
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    w, T = _dev(wl.wait_s, _f64()), _dev(wl.ctx_tokens, _i32())
    lp = _lib_prices(kvr, wl)
    sorted_ = method == kvr.KVR_SORTED
    if sorted_:
        ref, ref_perm = kvr.kvr_cost_grid(w, T, lp, g, method=method, want_perm=True)
    else:
        ref, ref_perm = kvr.kvr_cost_grid(w, T, lp, g, method=method), None
    perm = torch.empty(wl.n, dtype=torch.int32, device="cuda") if sorted_ else None
    cost, perm, status = kvr.kvr_cost_grid_noalloc(w, T, lp, g, method=method, perm=perm)
    torch.cuda.synchronize()
    assert int(_np(status)[0]) == kvr.KVR_OK
    return _np(cost), None if perm is None else _np(perm), _np(ref), \
        None if ref_perm is None else _np(ref_perm), g


@pytest.mark.parametrize("method", ["brute", "sorted"])
def test_noalloc_equals_cost_grid_twice(kvr, method):
    """Same plan as kvr_cost_grid, so bit-identical costs (and order); the
    second, smaller call follows on the scratch the first one left behind."""
    m = kvr.KVR_BRUTE if method == "brute" else kvr.KVR_SORTED
    for seed, n, k1, k2, L in ((501, 70000, 3, 70, 9), (502, 3000, 2, 20, 5)):
        wl = workloads.random_case(seed, n, k1, k2, L, ties=True)
        cost, perm, ref, ref_perm, _ = _both(kvr, wl, m)
        assert np.array_equal(cost, ref)
        if perm is not None:
            assert np.array_equal(perm, ref_perm)


def test_noalloc_small_sample_one_block_sort(kvr):
    """2,048 waits and fewer take the one-block sort: then 700 waits."""
    for seed, n in ((503, 2048), (504, 700)):
        wl = workloads.random_case(seed, n, 1, 65, 4, ties=True)
        cost, perm, ref, ref_perm, _ = _both(kvr, wl, kvr.KVR_SORTED)
        assert np.array_equal(cost, ref) and np.array_equal(perm, ref_perm)


def test_noalloc_fewer_splits_to_fit(kvr, oracle_mod):
    """weibull-1m by brute force: kvr_cost_grid's plan keeps 512 sample splits
    (269 MB of partials); in 64 MiB the same call sums fewer, larger splits.
    Costs within 1e-9 of kvr_cost_grid's, the same selections; then the tiny
    workload on the same scratch, bit-identical."""
    import torch
    wl = workloads.make("weibull-1m")
    cost, _, ref, _, g = _both(kvr, wl, kvr.KVR_BRUTE)
    assert_costs(cost, ref)
    b = _np(kvr.kvr_select_policy(torch.as_tensor(cost).cuda(), g.last_inf)[0])
    rb = _np(kvr.kvr_select_policy(torch.as_tensor(ref).cuda(), g.last_inf)[0])
    assert_selection(ref, b, rb)
    tiny = workloads.make("tiny-exp-1k")
    cost, _, ref, _, _ = _both(kvr, tiny, kvr.KVR_BRUTE)
    assert np.array_equal(cost, ref)


def test_noalloc_status_and_limit(kvr):
    """A NaN wait sets the status output to KVR_E_DOMAIN; the next clean call
    on the same scratch reports KVR_OK; a sample whose workspace exceeds the
    scratch is refused with KVR_E_SIZE before anything runs."""
    import torch
    wl = workloads.random_case(505, 5000, 2, 66, 3)
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    lp = _lib_prices(kvr, wl)
    w = wl.wait_s.copy()
    w[123] = np.nan
    T = _dev(wl.ctx_tokens, _i32())
    for method in (kvr.KVR_BRUTE, kvr.KVR_SORTED):
        _, _, status = kvr.kvr_cost_grid_noalloc(_dev(w, _f64()), T, lp, g, method=method)
        torch.cuda.synchronize()
        assert int(_np(status)[0]) == kvr.KVR_E_DOMAIN
        _, _, status = kvr.kvr_cost_grid_noalloc(_dev(wl.wait_s, _f64()), T, lp, g,
                                                 method=method)
        torch.cuda.synchronize()
        assert int(_np(status)[0]) == kvr.KVR_OK
    big = torch.zeros(1 << 21, dtype=torch.float64, device="cuda")
    bigT = torch.ones(1 << 21, dtype=torch.int32, device="cuda")
    with pytest.raises(kvr.KvrError) as ei:
        kvr.kvr_cost_grid_noalloc(big, bigT, lp, g, method=kvr.KVR_SORTED)
    assert ei.value.code == kvr.KVR_E_SIZE
