"""GPU parity on the second workload: the Section 4.1 families as three index
rows of one base sample, priced with each Table 3 vector (H100 NVL, A100 SXM,
L40S; beta_2 = 0.02, C2 = 425).  The bootstrap entry point (every policy of
every row, fused selection and the full cost tensor) and the SORTED path per
family against the oracle's closed form: costs within 1e-9 relative, the
selected policy identical up to rounding-level near ties; sampled host-timer
columns of both against the oracle's double loop."""
import numpy as np
import pytest

import workloads
from tests.test_gpu_parity import _dev, _f64, _i32, _np, assert_costs, assert_selection

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kvr():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2608_30830_amd as k
    k.load_library()
    return k


@pytest.fixture(scope="module")
def case():
    return workloads.cross_platform_case()


def _prices(kvr, platform):
    a1, b2, b3 = workloads.PLATFORM_PRICES[platform]
    p = kvr.kvr_prices_from_platform(1.0, 1.0, 1.0, 1.0, 1.0, 425.0, 1800.0)
    p.a1_per_token, p.b2_per_token, p.b3_per_token = a1, b2, b3
    return p


@pytest.mark.parametrize("platform", sorted(workloads.PLATFORM_PRICES))
def test_platform_bootstrap_rows(kvr, oracle_mod, case, platform):
    g = kvr.PolicyGrid(case.t1, case.t2, case.lam)
    best, bc, cost = kvr.kvr_bootstrap(_dev(case.wait_s, _f64()), _dev(case.ctx_tokens, _i32()),
                                       _dev(case.idx, _i32()), _prices(kvr, platform), g,
                                       want_cost=True)
    pr = oracle_mod.Prices(*workloads.PLATFORM_PRICES[platform])
    for r in range(3):
        ref = oracle_mod.closed_form_grid(case.wait_s, case.ctx_tokens, pr, case.t1, case.t2,
                                          case.lam, idx_row=case.idx[r])
        assert_costs(_np(cost)[r], ref)
        rb, rbc, _ = oracle_mod.select(ref, case.t2)
        assert_selection(ref, _np(best)[r], rb)
        assert_costs(_np(bc)[r], rbc)
        cols = np.array([0, 64, 150, case.t2.size - 2, case.t2.size - 1])
        loop = oracle_mod.cost_grid(case.wait_s, case.ctx_tokens, pr, case.t1, case.t2[cols],
                                    case.lam, idx_row=case.idx[r])
        assert_costs(_np(cost)[r][:, :, cols], loop)


@pytest.mark.parametrize("platform", sorted(workloads.PLATFORM_PRICES))
def test_platform_sorted_per_family(kvr, oracle_mod, case, platform):
    g = kvr.PolicyGrid(case.t1, case.t2, case.lam)
    pr = oracle_mod.Prices(*workloads.PLATFORM_PRICES[platform])
    n = case.m
    for r in range(3):
        w, T = case.wait_s[r * n:(r + 1) * n], case.ctx_tokens[r * n:(r + 1) * n]
        cost, perm = kvr.kvr_cost_grid(_dev(w, _f64()), _dev(T, _i32()), _prices(kvr, platform),
                                       g, method=kvr.KVR_SORTED, want_perm=True)
        ref = oracle_mod.closed_form_grid(w, T, pr, case.t1, case.t2, case.lam)
        assert_costs(_np(cost), ref)
        assert np.array_equal(_np(perm), oracle_mod.stable_order(w))
        # and sampled host-timer columns against the double loop
        cols = np.array([0, 37, 101, 180, case.t2.size - 2, case.t2.size - 1])
        loop = oracle_mod.cost_grid(w, T, pr, case.t1, case.t2[cols], case.lam)
        assert_costs(_np(cost)[:, :, cols], loop)
