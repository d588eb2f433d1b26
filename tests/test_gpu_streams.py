"""Every Python wrapper on a caller's side stream.

The wrappers return before the work they queue has finished, and the
workspace (and the outputs) they allocate belong to torch's caching
allocator.  Each call here runs on a side stream with the device check
deferred, while the current stream immediately allocates and overwrites
buffers of the same sizes; the results must equal, bit for bit, those of the
same call on the current stream (every path reduces in a fixed order).
"""
import numpy as np
import pytest

import workloads

pytestmark = pytest.mark.gpu

LC = 425.0 / 1800.0


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


def _np(t):
    return t.detach().cpu().numpy()


def _scribble(nbytes):
    """Allocate and overwrite current-stream memory while the side stream works."""
    import torch
    bufs = [torch.full((max(nbytes, 256) // 8,), float("nan"), dtype=torch.float64, device="cuda")
            for _ in range(4)]
    del bufs


def _side(fn):
    """Run fn(stream) on a fresh default-priority side stream, scribble, wait."""
    import torch
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    out = fn(s)
    _scribble(64 << 20)
    s.synchronize()
    return out


@pytest.fixture(scope="module")
def case(kvr):
    import torch
    wl = workloads.random_case(4242, 3001, 3, 70, 5, resamples=6)
    pf = wl.platform
    prices = kvr.kvr_prices_from_platform(wl.kv_bytes_per_token, pf["hbm_usable_bytes"],
                                          pf["host_link_bytes_per_s"],
                                          pf["prefill_tokens_per_s"], pf["n_gpu"],
                                          pf["host_slots_c2"], pf["w_ref_s"])
    return dict(w=_dev(wl.wait_s, torch.float64), T=_dev(wl.ctx_tokens, torch.int32),
                idx=_dev(wl.idx, torch.int32), prices=prices,
                grid=kvr.PolicyGrid(wl.t1, wl.t2, wl.lam))


@pytest.mark.parametrize("method", ["brute", "sorted"])
def test_cost_grid_side_stream(kvr, case, method):
    m = kvr.KVR_BRUTE if method == "brute" else kvr.KVR_SORTED
    perm = method == "sorted"
    ref = kvr.kvr_cost_grid(case["w"], case["T"], case["prices"], case["grid"], m, want_perm=perm)
    got = _side(lambda s: kvr.kvr_cost_grid(case["w"], case["T"], case["prices"], case["grid"], m,
                                            want_perm=perm, stream=s, check=False))
    if perm:
        np.testing.assert_array_equal(_np(got[1]), _np(ref[1]))
        got, ref = got[0], ref[0]
    np.testing.assert_array_equal(_np(got), _np(ref))


@pytest.mark.parametrize("factored", [False, True])
def test_bootstrap_side_stream(kvr, case, factored):
    args = (case["w"], case["T"], case["idx"], case["prices"], case["grid"])
    ref = kvr.kvr_bootstrap(*args, want_cost=True, factored=factored)
    got = _side(lambda s: kvr.kvr_bootstrap(*args, want_cost=True, factored=factored, stream=s,
                                            check=False))
    for g, r in zip(got, ref):
        np.testing.assert_array_equal(_np(g), _np(r))


def test_select_side_stream(kvr, case):
    cost = kvr.kvr_cost_grid(case["w"], case["T"], case["prices"], case["grid"])
    ref = kvr.kvr_select_policy(cost, True)
    got = _side(lambda s: kvr.kvr_select_policy(cost, True, stream=s))
    for g, r in zip(got, ref):
        np.testing.assert_array_equal(_np(g), _np(r))


def test_replay_and_controller_side_stream(kvr):
    import torch
    c2 = 40.0
    rc = workloads.replay_case("mixture", 3 * LC * c2 / 425.0, reps=3, n=2000, seed=77)
    p = kvr.kvr_prices_from_platform(1.0, 1.0, 1.0, 1.0, 1.0, c2, 1800.0)
    p.b2_per_token, p.b3_per_token = 0.02, 1.91
    arr, w = _dev(rc.arrival_s, torch.float64), _dev(rc.wait_s, torch.float64)
    t2 = [30.0, 600.0, float("inf")]
    ref = kvr.kvr_capacity_replay(arr, w, p, t2)
    got = _side(lambda s: kvr.kvr_capacity_replay(arr, w, p, t2, stream=s, check=False))
    for g, r in zip(got, ref):
        np.testing.assert_array_equal(_np(g), _np(r))

    lam = 3 * LC * c2 / 425.0
    ref_out = bytes(kvr.kvr_controller_select(arr, w, p, lam))

    def ctl(s):
        call = kvr.ControllerCall(arr, w, p, lam)
        call.launch(s)
        return call
    call = _side(ctl)
    assert bytes(call.result(torch.cuda.current_stream())) == ref_out


def test_crossover_side_stream(kvr, case):
    ref = kvr.kvr_crossover_statistic(case["w"], case["prices"])
    got = _side(lambda s: kvr.kvr_crossover_statistic(case["w"], case["prices"], stream=s,
                                                      check=False))
    for g, r in zip(got, ref):
        np.testing.assert_array_equal(_np(g), _np(r))
