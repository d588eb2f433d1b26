"""HIP-graph capture of prepared calls (the brute-force and the factored
bootstrap, the controller).  The entry points only enqueue kernels
on the caller's stream (no allocation, no memset, no synchronisation; the
host tables travel as kernel arguments), so a prepared BootstrapCall or
ControllerCall can be captured once and replayed.  Every replay, with eager
work on the same buffers in between, must give the eager result bit for
bit."""
import ctypes

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


@pytest.mark.parametrize("factored", [False, True])
def test_bootstrap_graph_replays(kvr, factored):
    import torch
    wl = workloads.make("boot-1024x64k", resamples=64)
    pf = wl.platform
    pr = kvr.kvr_prices_from_platform(wl.kv_bytes_per_token, pf["hbm_usable_bytes"],
                                      pf["host_link_bytes_per_s"], pf["prefill_tokens_per_s"])
    g = kvr.PolicyGrid(wl.t1, wl.t2, wl.lam)
    call = kvr.BootstrapCall(torch.as_tensor(wl.wait_s).cuda(), torch.as_tensor(wl.ctx_tokens).cuda(),
                             torch.as_tensor(wl.idx).cuda(), pr, g, want_cost=True,
                             factored=factored)
    call.launch()
    torch.cuda.synchronize()
    assert call.status() == kvr.KVR_OK
    ref = (call.best.clone(), call.best_cost.clone(), call.cost.clone())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call.launch()
    for _ in range(3):
        call.best.fill_(-7)                     # eager work on the outputs between replays
        call.best_cost.fill_(0.0)
        call.cost.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert call.status() == kvr.KVR_OK
        assert torch.equal(call.best, ref[0])
        assert torch.equal(call.best_cost, ref[1])
        assert torch.equal(call.cost, ref[2])


def test_controller_graph_replays(kvr):
    import torch
    rc = workloads.replay_case("mixture", 2 * LC, reps=256, n=4000, seed=5)
    p = kvr.kvr_prices_from_platform(1.0, 1.0, 1.0, 1.0, 1.0, 425.0, 1800.0)
    p.a1_per_token, p.b2_per_token, p.b3_per_token = 0.0176, 0.02, 1.91
    call = kvr.ControllerCall(torch.as_tensor(rc.arrival_s).cuda(), torch.as_tensor(rc.wait_s).cuda(),
                              p, 2 * LC)
    call.launch()
    ref = bytes(call.result())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call.launch()
    for _ in range(3):
        call.out.fill_(0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert bytes(call.result()) == ref
