"""Pins of the second workload: the Section 4.1 wait families priced with the
three Table 3 price vectors (cross-platform calibration, Appendix C).

The oracle's closed form (itself pinned against the double loop) evaluates
every (family, platform); what the paper fixes is checked on it: below
lambda_crit host capacity does not bind and the selection is host-retain
with offload at suspension, costing exactly beta_2; and for exponential
waits well above the memoryless threshold the earliest timer wins on every
platform."""
import numpy as np
import pytest

import workloads

LC = 425.0 / 1800.0


@pytest.fixture(scope="module")
def case():
    return workloads.cross_platform_case()


def _family(wl, r):
    n = wl.m
    return wl.wait_s[r * n:(r + 1) * n], wl.ctx_tokens[r * n:(r + 1) * n]


@pytest.mark.parametrize("platform", sorted(workloads.PLATFORM_PRICES))
def test_uncongested_selects_retain_at_beta2(oracle_mod, case, platform):
    a1, b2, b3 = workloads.PLATFORM_PRICES[platform]
    pr = oracle_mod.Prices(a1, b2, b3)
    K2 = case.t2.size
    for r, family in enumerate(workloads.FAMILIES):
        w, T = _family(case, r)
        cost = oracle_mod.closed_form_grid(w, T, pr, case.t1, case.t2, case.lam)
        best, bc, branch = oracle_mod.select(cost, case.t2)
        for l, lam in enumerate(case.lam):
            if lam <= LC:
                assert best[l] == K2 - 1, (platform, family, lam)   # t1 = 0, t2 = inf
                assert branch[l] == 0
                assert abs(bc[l] - b2) <= 1e-15


@pytest.mark.parametrize("platform", sorted(workloads.PLATFORM_PRICES))
def test_exponential_well_above_threshold_expires_first(oracle_mod, case, platform):
    """Memoryless waits: retain wins iff lambda <= lambda_crit + C2 (1 - b2/b3)/mu
    (about 0.47/s for all three vectors); at 3 lambda_crit = 0.71/s the
    shortest host timer of the grid is chosen, with offload at suspension."""
    a1, b2, b3 = workloads.PLATFORM_PRICES[platform]
    thr = LC + 425.0 * (1.0 - b2 / b3) / 1800.0
    assert 0.46 < thr < 0.48
    pr = oracle_mod.Prices(a1, b2, b3)
    w, T = _family(case, workloads.FAMILIES.index("exponential"))
    cost = oracle_mod.closed_form_grid(w, T, pr, case.t1, case.t2, case.lam)
    best, _, branch = oracle_mod.select(cost, case.t2)
    l3 = int(np.argmax(case.lam))
    assert case.lam[l3] == pytest.approx(3 * LC) and case.lam[l3] > thr
    assert best[l3] == 0 and branch[l3] == 1


def test_rows_are_the_families(case):
    assert case.idx.shape == (3, case.m)
    for r in range(3):
        assert np.array_equal(case.idx[r], np.arange(r * case.m, (r + 1) * case.m))
        w, T = _family(case, r)
        assert abs(w.mean() - 1800.0) < 40.0 and np.all(T == 1)
