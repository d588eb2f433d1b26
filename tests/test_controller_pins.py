"""Pins of the oracle's regime-aware controller (Section 3.4, frozen across
loads as in Appendix F) and of the crossover statistic P(W <= t*) (Section
4.3, Figure 4(d), the last column of Table 3).

The controller is pinned against an exact composition of the list-based
replay, the degenerate load at or below lambda_crit, the branches Table 6
prints, and the crossover values Table 3 prints for three platforms; the
statistic against closed-form population shares of the synthetic wait
distributions and the boundary w = t*."""
import math
from fractions import Fraction

import numpy as np
import pytest

import workloads
from oracle import exact
from tests import helpers as H
from tests.test_replay_pins import _table6, _tiny

LC = 425.0 / 1800.0
B2, B3, A1 = 0.02, 1.91, 0.0176          # per request, H100 NVL (Appendix B, Table 3)


def _lam_for_timer(c2, t2, b2=B2, b3=B3, w_ref=1800.0):
    """The load at which the Eq. 3 timer is t2."""
    return c2 / w_ref + (b3 - b2) / t2 * c2 / b3


@pytest.mark.parametrize("seed", range(16))
@pytest.mark.parametrize("c2", [1, 2, 3])
def test_controller_is_the_exact_two_branch_replay(oracle_mod, seed, c2):
    """Totals and counts equal those of the exact list simulation run under
    both branches; the branch is the cheaper exact total (retain on ties)."""
    arr, w, T = _tiny(seed)
    lam = _lam_for_timer(c2, 12.0)
    out = oracle_mod.controller_select(arr, w, c2, lam, A1, B2, B3, ctx=T)
    t2 = oracle_mod.eq3_timer(lam, B2, B3, float(c2), 1800.0)
    assert out.t2_s == t2 and abs(t2 - 12.0) < 1e-9
    tot = int(T.sum())
    exact_total = []
    for k, timer in enumerate((t2, math.inf)):
        _, rest, adm = exact.capacity_replay(arr, w, c2, timer, B2, B3, ctx=T)
        assert (rest, adm) == ((out.restored_timer, out.admitted_timer),
                               (out.restored_retain, out.admitted_retain))[k]
        exact_total.append(Fraction(B2) * rest + Fraction(B3) * (tot - rest))
    got = (out.total_cost_timer, out.total_cost_retain)
    for k in range(2):
        assert abs(got[k] - float(exact_total[k])) <= 2 * H.EPS * float(exact_total[k])
    assert out.total_tokens == tot and out.n_requests == w.size
    if exact_total[0] != exact_total[1]:
        assert out.branch == (1 if exact_total[0] < exact_total[1] else 0)


@pytest.mark.parametrize("mult", [0.0, 0.5, 1.0])
def test_controller_at_or_below_lambda_crit_keeps_retain(oracle_mod, mult):
    """At or below lambda_crit the Eq. 3 timer is infinite: both branches are
    host-retain, the totals are equal and the tie keeps retain."""
    rc = workloads.replay_case("mixture", max(mult, 0.25) * LC, reps=4, n=2000, seed=3)
    out = oracle_mod.controller_select(rc.arrival_s, rc.wait_s, 425, mult * LC, A1, B2, B3)
    assert math.isinf(out.t2_s)
    assert out.total_cost_timer == out.total_cost_retain
    assert out.restored_timer == out.restored_retain
    assert out.branch == 0


@pytest.mark.parametrize("family", workloads.FAMILIES)
def test_controller_freezes_table6_branch(oracle_mod, family):
    """Table 6: calibrated once at 2 lambda_crit on a sample disjoint from the
    held-out replays, the controller keeps host-retain for lognormal and
    exponential waits and the Eq. 3 timer for the mixture."""
    rows, _ = _table6()
    rc = workloads.replay_case(family, 2 * LC, reps=64, seed=77)
    out = oracle_mod.controller_select(rc.arrival_s, rc.wait_s, 425, 2 * LC, A1, B2, B3)
    assert ("ttl" if out.branch == 1 else "retain") == rows[(family, 2.0)][1]


# Table 3: (platform, alpha_1, beta_3, printed t*, printed crossover P(W <= t*)).
TABLE3 = [("H100 NVL", 0.0176, 1.91, 109.0, 0.39),
          ("A100 SXM", 0.0232, 2.61, 112.0, 0.39),
          ("L40S", 0.118, 5.14, 43.5, 0.23)]


def crossover_sweep(oracle_mod, a1, b3, weights, reps=60):
    """Figure 4(d) as a sweep: the mixture's share of short approvals varies
    (mean wait held at 1,800 s); at 2 lambda_crit each point gives the gain of
    the Eq. 3 timer over host-retain (positive favours expiration) and the
    calibration sample's P(W <= t*)."""
    pts = []
    for q in weights:
        rc = workloads.replay_case("mixture", 2 * LC, reps=reps, seed=404, short_weight=q)
        out = oracle_mod.controller_select(rc.arrival_s, rc.wait_s, 425, 2 * LC, a1, B2, b3)
        pts.append((out.p_short, out.total_cost_retain / out.total_cost_timer - 1.0, out.branch))
    return pts


def crossing(pts):
    """P(W <= t*) where the gain first changes sign (linear interpolation)."""
    for (p0, g0, _), (p1, g1, _) in zip(pts, pts[1:]):
        if g0 < 0.0 <= g1:
            return p0 + (p1 - p0) * (-g0) / (g1 - g0)
    return None


@pytest.mark.parametrize("platform,a1,b3,t_star,printed", TABLE3)
def test_crossover_matches_table3(oracle_mod, platform, a1, b3, t_star, printed):
    """The break-even time t* = beta_3 / alpha_1 is the printed one (3
    significant figures) and the gain of the timer over retain changes sign
    at the printed P(W <= t*) within 0.03; the frozen branch follows the sign
    of the gain at every point."""
    assert abs(b3 / a1 - t_star) <= 0.006 * t_star
    pts = crossover_sweep(oracle_mod, a1, b3, np.linspace(0.2, 0.7, 11))
    assert pts[0][1] < 0.0 < pts[-1][1], pts
    x = crossing(pts)
    assert x is not None and abs(x - printed) <= 0.03, (platform, x, pts)
    for p, g, br in pts:
        assert br == (1 if g > 0.0 else 0)


def _lognormal_cdf(t, median, sigma):
    return 0.5 * math.erfc(-(math.log(t) - math.log(median)) / (sigma * math.sqrt(2.0)))


def _weibull_trunc_cdf(t, shape=0.5, scale=1800.0, cap=86400.0):
    return -math.expm1(-(t / scale) ** shape) / -math.expm1(-(cap / scale) ** shape)


POPULATION = {
    "tiny-exp-1k": lambda t: -math.expm1(-t / 1800.0),
    "mix-64k": lambda t: 0.7 * _lognormal_cdf(t, 60.0, 1.0) + 0.3 * _lognormal_cdf(t, 7200.0, 0.8),
    "weibull-1m": _weibull_trunc_cdf,
}


@pytest.mark.parametrize("name,expect", [("tiny-exp-1k", 0.052), ("mix-64k", 0.475),
                                         ("weibull-1m", 0.136)])
def test_crossover_share_of_the_workloads(oracle_mod, name, expect):
    """On each workload the sample share of waits at or below its own t*
    lies within 4 binomial standard deviations of the population share of
    its wait law, which is the value quoted for that workload."""
    wl = workloads.make(name)
    pr = oracle_mod.workload_prices(wl)
    t_star = pr.b3 / pr.a1
    pop = POPULATION[name](t_star)
    assert abs(pop - expect) < 0.0015, (name, pop)
    share = oracle_mod.crossover_count(wl.wait_s, pr.a1, pr.b3) / wl.n
    assert abs(share - pop) <= 4.0 * math.sqrt(pop * (1.0 - pop) / wl.n), (name, share, pop)


def test_crossover_counts_the_break_even_wait(oracle_mod):
    """A wait equal to t* counts (W <= t*); the next double above does not."""
    a1, b3 = 0.0232, 2.61
    t_star = b3 / a1
    w = np.array([0.0, t_star, np.nextafter(t_star, np.inf), 1e6, t_star / 2])
    assert oracle_mod.crossover_count(w, a1, b3) == 3
    arr = np.arange(w.size, dtype=np.float64)
    out = oracle_mod.controller_select(arr, w, 2, 2 * LC, a1, B2, b3)
    assert out.n_short == 3 and out.p_short == 3 / 5 and out.t_star_s == t_star


def test_controller_sample_statistic_is_the_crossover_count(oracle_mod):
    rc = workloads.replay_case("lognormal", 2 * LC, reps=8, n=1000, seed=12)
    out = oracle_mod.controller_select(rc.arrival_s, rc.wait_s, 425, 2 * LC, A1, B2, B3)
    assert out.n_short == oracle_mod.crossover_count(rc.wait_s, A1, B3)
    assert out.n_requests == 8000 and out.p_short == out.n_short / 8000


def _meanfield_two_branch(oracle_mod, w, lam):
    """The two branches of Section 3.4 priced by the mean-field cost of the
    grid (Eq. 1 with the Eq. 3 congestion price, offload at suspension):
    [cost of the Eq. 3 timer t2(lambda), cost of retain]."""
    t2 = oracle_mod.eq3_timer(lam, B2, B3, 425.0, 1800.0)
    pr = oracle_mod.Prices(A1, B2, B3)
    T = np.ones(w.size, np.int32)
    cost = oracle_mod.cost_grid(w, T, pr, np.array([0.0]), np.array([t2, np.inf]),
                                np.array([lam]))
    return cost[0, 0], t2


def test_meanfield_two_branch_closed_form(oracle_mod):
    """Exponential waits (mean mu): retain costs b2 + a2 mu and the timer
    b2 + (b3 - b2) exp(-t2/mu) + a2 mu (1 - exp(-t2/mu)) with
    a2 = (lambda - lambda_crit) b3 / C2; at 2 lambda_crit that is 1.9226
    against 1.9300, so the mean-field comparison takes the timer."""
    w = H.stratified_exponential(200000, 1800.0)
    (c_ttl, c_ret), t2 = _meanfield_two_branch(oracle_mod, w, 2 * LC)
    a2 = (2 * LC - LC) * B3 / 425.0
    s = math.exp(-t2 / 1800.0)
    assert abs(c_ret - (B2 + a2 * 1800.0)) < 2e-3
    assert abs(c_ttl - (B2 + (B3 - B2) * s + a2 * 1800.0 * (1.0 - s))) < 2e-3
    assert abs(c_ttl - 1.9226) < 2e-3 and abs(c_ret - 1.930) < 2e-3


@pytest.mark.parametrize("family", workloads.FAMILIES)
def test_meanfield_and_replay_controllers_disagree_above_lambda_crit(oracle_mod, family):
    """At 2 lambda_crit the mean-field cost prefers the Eq. 3 timer for all
    three families, while the finite-capacity replay (the paper's controller,
    Table 6) keeps retain for lognormal and exponential waits: the congestion
    price is a mean-field reading that the replay does not charge."""
    (c_ttl, c_ret), _ = _meanfield_two_branch(oracle_mod, H.stratified_family(family, 100000),
                                              2 * LC)
    assert c_ttl < c_ret
    rows, _ = _table6()
    rc = workloads.replay_case(family, 2 * LC, reps=64, seed=77)
    out = oracle_mod.controller_select(rc.arrival_s, rc.wait_s, 425, 2 * LC, A1, B2, B3)
    assert ("ttl" if out.branch == 1 else "retain") == rows[(family, 2.0)][1]
    assert (out.branch == 1) == (family == "mixture")
