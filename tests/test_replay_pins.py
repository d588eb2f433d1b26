"""Pins of the oracle's finite-capacity admission replay (Appendix D, the
evaluation behind Tables 3 and 6) against an independent list-based
simulation, the no-contention limit of the cost grid, the Erlang loss formula,
and the paper's printed replay results."""
import math

import numpy as np
import pytest

import workloads
from oracle import exact
from tests import helpers as H

LC = 425.0 / 1800.0


def _tiny(seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    n = int(rng.integers(1, 40))
    arr = np.cumsum(rng.exponential(3.0, n))
    w = rng.exponential(20.0, n)
    if n > 6:
        arr[3] = arr[2]                      # simultaneous arrivals
        w[4] = arr[5] - arr[4]               # a resume exactly at a later arrival
        w[1] = 0.0                           # resume at suspension
        w[6] = 7.5                           # a wait exactly on a timer
    T = rng.integers(1, 9, n).astype(np.int32)
    return arr, w, T


@pytest.mark.parametrize("seed", range(16))
@pytest.mark.parametrize("c2", [1, 2, 3, 7])
@pytest.mark.parametrize("t2", [7.5, 30.0, math.inf])
def test_replay_matches_list_simulation(oracle_mod, seed, c2, t2):
    arr, w, T = _tiny(seed)
    cost, rest, adm = oracle_mod.capacity_replay(arr, w, c2, t2, 0.02, 1.91, ctx=T)
    ec, er, ea = exact.capacity_replay(arr, w, c2, t2, 0.02, 1.91, ctx=T)
    assert (rest, adm) == (er, ea)
    assert abs(cost - float(ec)) <= 2 * H.EPS * abs(float(ec))


def test_replay_without_contention_is_the_uncongested_grid(oracle_mod):
    """With C2 at least the number of requests nobody is refused, so the
    replay cost is the grid's cost at t1 = 0 below lambda_crit (no holding
    price): the mean of T * (w <= t2 ? b2 : b3)."""
    rng = np.random.Generator(np.random.PCG64(3))
    n = 3000
    w = rng.lognormal(6.0, 1.5, n)
    arr = np.cumsum(rng.exponential(1.0, n))
    T = rng.integers(1, 5000, n).astype(np.int32)
    pr = oracle_mod.Prices(1e-6, 2e-6, 5e-5, 425.0, 1800.0)
    t2 = np.array([60.0, 600.0, 3600.0, np.inf])
    grid = oracle_mod.cost_grid(w, T, pr, np.array([0.0]), t2, np.array([0.1]))[0, 0]
    for k, t in enumerate(t2):
        cost, _, adm = oracle_mod.capacity_replay(arr, w, n, t, pr.b2, pr.b3, ctx=T)
        assert adm == n
        assert abs(cost - grid[k]) <= 1e-12 * grid[k]


def _erlang_b(c, rho):
    b = 1.0
    for k in range(1, c + 1):
        b = rho * b / (k + rho * b)
    return b


@pytest.mark.parametrize("family,t2", [("exponential", math.inf), ("lognormal", math.inf),
                                       ("exponential", 1200.0), ("mixture", 2400.0)])
def test_replay_steady_state_is_erlang_loss(oracle_mod, family, t2):
    """Poisson arrivals into C2 slots that each hold a context for min(W, t2):
    an M/G/c/c loss system, whose blocking is the Erlang B formula for
    rho = lambda E[min(W, t2)] whatever the holding law; by PASTA the
    restored share is (1 - B) P(W <= t2).  A long run (200,000 requests)
    makes the empty start negligible."""
    c2 = 120
    rng = np.random.Generator(np.random.PCG64(11))
    w = workloads.family_waits(rng, family, 200000)
    hold = np.minimum(w, t2).mean()          # the sample's own mean holding time
    lam = 1.3 * c2 / hold                    # 30 % overload
    arr = np.cumsum(rng.exponential(1.0 / lam, w.size))
    cost, rest, adm = oracle_mod.capacity_replay(arr, w, c2, t2, 0.0, 1.0)
    B = _erlang_b(c2, lam * hold)
    share_restored = rest / w.size
    expect = (1.0 - B) * np.mean(w <= t2)
    assert abs(share_restored - expect) < 0.01, (share_restored, expect, B)
    assert abs((1.0 - adm / w.size) - B) < 0.01


def _table6():
    rows = {}
    table3 = []
    for r in H.read_table("table6_load_sweep.txt"):
        if r[0] == "TABLE3":
            table3.append((r[1], float(r[2]), [float(x) for x in r[3:6]]))
        else:
            rows[(r[0], float(r[1]))] = ([float(x) for x in r[2:7]], r[7])
    return rows, table3


@pytest.mark.parametrize("family", workloads.FAMILIES)
def test_table6_within_replay_spread(oracle_mod, family):
    """Table 6: every printed cell lies within 3.5 standard deviations (of one
    4,000-request replay) of the mean over 100 replays; the fixed-timer and
    retain columns below lambda_crit within 0.03 of it."""
    rows, _ = _table6()
    for mult in (0.5, 1.0, 2.0, 3.0):
        lam = mult * LC
        ttl = oracle_mod.eq3_timer(lam, 0.02, 1.91, 425.0, 1800.0)
        t2 = np.array([ttl, np.inf, 600.0, 1800.0, 3600.0])
        rc = workloads.replay_case(family, lam, reps=100)
        cost, _ = oracle_mod.capacity_replay_batch(rc.arrival_s, rc.wait_s, 425, t2, 0.02, 1.91)
        mean, sd = cost.mean(0), cost.std(0)
        printed, _ = rows[(family, mult)]
        for j in range(5):
            assert abs(printed[j] - mean[j]) <= 3.5 * sd[j] + 0.03, (family, mult, j, printed[j],
                                                                     mean[j], sd[j])


@pytest.mark.parametrize("family", workloads.FAMILIES)
def test_table6_controller_branch(oracle_mod, family):
    """Section 3.4 / Table 6: replaying calibration waits under both host
    branches at the reference load 2 lambda_crit and keeping the cheaper one
    selects host-retain for lognormal and exponential waits and the Eq. 3
    timer for the mixture, as the controller column prints."""
    rows, _ = _table6()
    lam = 2 * LC
    ttl = oracle_mod.eq3_timer(lam, 0.02, 1.91, 425.0, 1800.0)
    rc = workloads.replay_case(family, lam, reps=64, seed=77)   # a calibration sample
    cost, _ = oracle_mod.capacity_replay_batch(rc.arrival_s, rc.wait_s, 425,
                                               np.array([ttl, np.inf]), 0.02, 1.91)
    pick = "ttl" if cost[:, 0].mean() < cost[:, 1].mean() else "retain"
    assert pick == rows[(family, 2.0)][1]


def test_table3_relative_cost_of_ttl(oracle_mod):
    """Table 3 replay columns: relative cost of cpu_ttl vs host-retain at
    2 lambda_crit with each platform's beta_3 (beta_2 = 0.02, C2 = 425):
    the sign of every entry and its size within 4 points."""
    _, table3 = _table6()
    lam = 2 * LC
    for platform, beta3, rel in table3:
        ttl = oracle_mod.eq3_timer(lam, 0.02, beta3, 425.0, 1800.0)
        for family, printed in zip(workloads.FAMILIES, rel):
            rc = workloads.replay_case(family, lam, reps=100, seed=5)
            cost, _ = oracle_mod.capacity_replay_batch(rc.arrival_s, rc.wait_s, 425,
                                                       np.array([ttl, np.inf]), 0.02, beta3)
            ours = 100.0 * (cost[:, 0].mean() / cost[:, 1].mean() - 1.0)
            assert np.sign(ours) == np.sign(printed), (platform, family, ours, printed)
            assert abs(ours - printed) <= 4.0, (platform, family, ours, printed)
