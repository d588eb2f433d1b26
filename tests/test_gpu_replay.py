"""GPU parity of the finite-capacity admission replay (kvr_capacity_replay)
against the oracle: restored tokens and admitted counts bit-exact, mean costs
within 4 ulps (the same formula, possibly contracted on the GPU)."""
import math

import numpy as np
import pytest

import workloads
from tests.test_replay_pins import _tiny

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


def _prices(kvr, b2=0.02, b3=1.91, c2=425.0):
    p = kvr.kvr_prices_from_platform(1.0, 1.0, 1.0, 1.0, 1.0, c2, 1800.0)
    p.b2_per_token, p.b3_per_token = b2, b3
    return p


def _run(kvr, arr, w, t2, c2, T=None, b2=0.02, b3=1.91):
    import torch
    cost, rest, adm = kvr.kvr_capacity_replay(_dev(arr, torch.float64), _dev(w, torch.float64),
                                              _prices(kvr, b2, b3, float(c2)), list(t2),
                                              ctx_tokens=None if T is None else _dev(T, torch.int32))
    return cost.cpu().numpy(), rest.cpu().numpy(), adm.cpu().numpy()


def _check(kvr, oracle_mod, arr, w, t2, c2, T=None):
    arr, w = np.atleast_2d(arr), np.atleast_2d(w)
    Tm = None if T is None else np.atleast_2d(T)
    cost, rest, adm = _run(kvr, arr, w, t2, c2, Tm)
    for r in range(arr.shape[0]):
        for k, t in enumerate(t2):
            oc, orr, oa = oracle_mod.capacity_replay(arr[r], w[r], c2, t, 0.02, 1.91,
                                                     ctx=None if Tm is None else Tm[r])
            assert (rest[r, k], adm[r, k]) == (orr, oa), (r, k, t)
            assert abs(cost[r, k] - oc) <= 4 * np.spacing(oc)


@pytest.mark.parametrize("seed", range(16))
def test_replay_tiny_crafted(kvr, oracle_mod, seed):
    arr, w, T = _tiny(seed)
    for c2 in (1, 2, 3, 7):
        _check(kvr, oracle_mod, arr, w, [7.5, 30.0, math.inf], c2, T)


@pytest.mark.parametrize("n", [1, 31, 32, 33, 1000, 4000, 8192])
@pytest.mark.parametrize("c2", [1, 17, 425])
def test_replay_ragged_sizes(kvr, oracle_mod, n, c2):
    rc = workloads.replay_case("mixture", 3 * LC * c2 / 425.0, reps=3, n=n, seed=31)
    _check(kvr, oracle_mod, rc.arrival_s, rc.wait_s, [60.0, 900.0, 3600.0, math.inf], c2)


@pytest.mark.parametrize("family", workloads.FAMILIES)
def test_replay_table6_conditions(kvr, oracle_mod, family):
    """The Table 6 grid (4 loads x Eq. 3 timer, retain, 10/30/60 min) over 256
    replays of 4,000 requests: every count identical to the oracle's."""
    for mult in (0.5, 1.0, 2.0, 3.0):
        lam = mult * LC
        ttl = oracle_mod.eq3_timer(lam, 0.02, 1.91, 425.0, 1800.0)
        t2 = np.array([ttl, np.inf, 600.0, 1800.0, 3600.0])
        rc = workloads.replay_case(family, lam, reps=256)
        cost, rest, adm = _run(kvr, rc.arrival_s, rc.wait_s, t2, 425)
        oc, orr = oracle_mod.capacity_replay_batch(rc.arrival_s, rc.wait_s, 425, t2, 0.02, 1.91)
        assert np.array_equal(rest, orr)
        assert np.all(np.abs(cost - oc) <= 4 * np.spacing(oc))


def test_replay_with_context_tokens(kvr, oracle_mod):
    rc = workloads.replay_case("lognormal", 2 * LC, reps=4, n=3000, seed=8)
    T = np.random.Generator(np.random.PCG64(2)).integers(1, 30000, rc.arrival_s.shape).astype(np.int32)
    _check(kvr, oracle_mod, rc.arrival_s, rc.wait_s, [1781.0, math.inf], 425, T)


def test_replay_domain_errors(kvr):
    import torch
    rc = workloads.replay_case("exponential", LC, reps=2, n=500, seed=4)
    for what in ("order", "nan", "neg"):
        arr, w = rc.arrival_s.copy(), rc.wait_s.copy()
        if what == "order":
            arr[1, 100] = arr[1, 99] - 1.0
        elif what == "nan":
            w[0, 7] = np.nan
        else:
            w[1, 3] = -2.0
        with pytest.raises(kvr.KvrError) as ei:
            kvr.kvr_capacity_replay(_dev(arr, torch.float64), _dev(w, torch.float64),
                                    _prices(kvr), [600.0, math.inf])
        assert ei.value.code == kvr.KVR_E_DOMAIN


def test_replay_many_timers_in_chunks(kvr, oracle_mod):
    """40 timers on 2,048 sequences of 8,192 requests exceed what one pass of
    the expiry words holds (1 GiB), so the timers run in two chunks; every
    count still equals the oracle's."""
    rc = workloads.replay_case("mixture", 3 * LC, reps=2048, n=8192, seed=91)
    t2 = np.concatenate([np.geomspace(30.0, 86400.0, 39), [np.inf]])
    cost, rest, adm = _run(kvr, rc.arrival_s, rc.wait_s, t2, 425)
    oc, orr = oracle_mod.capacity_replay_batch(rc.arrival_s, rc.wait_s, 425, t2, 0.02, 1.91)
    assert np.array_equal(rest, orr)
    assert np.all(np.abs(cost - oc) <= 4 * np.spacing(oc))


@pytest.mark.parametrize("reps,n,n_timers", [(4096, 2500, 9), (4096, 5000, 5)])
def test_replay_forty_lane_waves(kvr, oracle_mod, reps, n, n_timers):
    """Batches whose (timer, sequence) lanes would need a second round of
    64-lane waves (LDS holds two per CU) run as 40-lane waves, four per CU:
    36,864 lanes with up to 4,096 requests per sequence, 20,480 with up to
    8,192.  Sampled rows against the oracle, every row's admissions within
    their bounds."""
    rc = workloads.replay_case("lognormal", 2 * LC, reps=reps, n=n, seed=123)
    t2 = np.concatenate([np.geomspace(60.0, 20000.0, n_timers - 1), [np.inf]])
    cost, rest, adm = _run(kvr, rc.arrival_s, rc.wait_s, t2, 425)
    rows = np.unique(np.linspace(0, reps - 1, 61).astype(int))
    oc, orr = oracle_mod.capacity_replay_batch(rc.arrival_s[rows], rc.wait_s[rows], 425, t2,
                                               0.02, 1.91)
    assert np.array_equal(rest[rows], orr)
    assert np.all(np.abs(cost[rows] - oc) <= 4 * np.spacing(oc))
    assert np.all((adm >= np.minimum(n, 425)) & (adm <= n))
    assert np.all(rest <= adm)
