"""The oracle's pins are strong enough to catch plausible mistakes.

Each mutant is a copy of the oracle's C source with one planted mistake (a
dropped term, a swapped price, a wrong boundary, a wrong sign or index),
compiled on the CPU into a temporary library.  The exact event simulation and
the closed-form expectation pins are run against it, and at least one of them
must fail.  Nothing here runs on a GPU.
"""
import ctypes
import os

import numpy as np
import pytest

import oracle
from oracle import exact
from tests import helpers as H
from tests.test_oracle_pins import _tiny_cases

SRC = os.path.join(os.path.dirname(oracle.__file__), "kvr_oracle.c")

MUTANTS = {
    "drop_host_holding": ("double host = a2 * (host_end - t1);", "double host = 0.0 * (host_end - t1);"),
    "swap_restore_recompute": ("(w <= e) ? b2 : b3;", "(w <= e) ? b3 : b2;"),
    "strict_deadline": ("(w <= e) ? b2 : b3;", "(w < e) ? b2 : b3;"),
    "hbm_full_t1": ("double hbm_time = (w < t1) ? w : t1;", "double hbm_time = t1;"),
    "host_sign": ("(host_end - t1)", "(host_end + t1)"),
    "lambda_crit_inverted": ("return c2 / w_ref;", "return w_ref / c2;"),
    "offload_at_equal": ("if (w > t1) {                                  /* offloaded at t1       */",
                         "if (w >= t1) {"),
    "tie_to_smaller": ("if (row[f] <= bc)", "if (row[f] < bc)"),
    "deadline_from_zero": ("double e = t1[a] + t2[k];\n        nsum acc", "double e = t2[k];\n        nsum acc"),
    "divide_by_n": ("cost_out[p] = nsum_get(&acc) / (double)m;", "cost_out[p] = nsum_get(&acc) / (double)(m + 1);"),
    "offload_charge_dropped": ("(host + resume + boff)", "(host + resume)"),
    "offload_charge_in_hbm": ("double cost = a1 * hbm_time;", "double cost = a1 * hbm_time + boff;"),
}


def _pins_pass(mod):
    """The exact-simulation cases, a two-tier bootstrap case, and the
    uncongested expectation pin; returns False at the first failure."""
    for pr in (mod.Prices(0.0524288, 0.0262144, 5e-5, 425.0, 1800.0),
               mod.Prices(0.0524288, 0.0262144, 5e-5, 425.0, 1800.0, boff=0.0131072)):
        for (w, T, t1, t2, lam) in _tiny_cases():
            got = mod.cost_grid(w, T, pr, t1, t2, lam)
            ex = np.array(exact.cost_grid(w, T, pr, t1, t2, lam), dtype=float)
            if not np.allclose(got, ex, rtol=4 * len(w) * H.EPS, atol=0):
                return False
            if list(np.atleast_1d(mod.select(got, t2)[0])) != exact.select(
                    exact.cost_grid(w, T, pr, t1, t2, lam)):
                return False
    w = H.stratified_family("exponential", 20000)
    c = mod.cost_grid(w, np.ones(w.size, np.int32), mod.Prices(0.0176, 0.02, 1.91),
                      np.array([0.0]), np.array([600.0, np.inf]), np.array([0.1]))
    expect = 0.02 + 1.89 * H.survival("exponential", 600.0)
    return abs(c[0, 0, 0] - expect) < 1e-3 and abs(c[0, 0, 1] - 0.02) < 1e-12


def test_unmutated_oracle_passes(oracle_mod):
    assert _pins_pass(oracle_mod)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(oracle_mod, tmp_path, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    mpath = tmp_path / "mutant.c"
    mpath.write_text(src.replace(old, new))
    lib = tmp_path / "libmutant.so"
    oracle.compile_library(str(mpath), str(lib))
    saved = oracle._lib
    try:
        oracle._lib = oracle._configure(ctypes.CDLL(str(lib)))
        assert not _pins_pass(oracle), f"mutant {name} survived the pins"
    finally:
        oracle._lib = saved


REPLAY_MUTANTS = {
    "expiry_never_frees": ("heap_push(&h, a + t2);", "heap_push(&h, a + w);"),
    "admit_one_short": ("if (h.size < c2) {", "if (h.size + 1 < c2 || h.size == 0) {"),
    "departure_strict": ("while (h.size > 0 && h.v[0] <= a) heap_pop(&h);",
                         "while (h.size > 0 && h.v[0] < a) heap_pop(&h);"),
    "timer_strict": ("if (w <= t2) {                                   /* resumes before the timer */",
                     "if (w < t2) {"),
}


def _replay_pins_pass(mod):
    from tests.test_replay_pins import _tiny
    for seed in range(16):
        arr, w, T = _tiny(seed)
        for c2 in (1, 2, 3):
            for t2 in (7.5, 30.0, float("inf")):
                got = mod.capacity_replay(arr, w, c2, t2, 0.02, 1.91, ctx=T)
                ref = exact.capacity_replay(arr, w, c2, t2, 0.02, 1.91, ctx=T)
                if got[1:] != ref[1:]:
                    return False
    return True


@pytest.mark.parametrize("name", sorted(REPLAY_MUTANTS))
def test_replay_mutant_is_caught(oracle_mod, tmp_path, name):
    old, new = REPLAY_MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    mpath = tmp_path / "mutant.c"
    mpath.write_text(src.replace(old, new))
    lib = tmp_path / "libmutant.so"
    oracle.compile_library(str(mpath), str(lib))
    saved = oracle._lib
    try:
        oracle._lib = oracle._configure(ctypes.CDLL(str(lib)))
        assert _replay_pins_pass(oracle) is False, f"mutant {name} survived"
    finally:
        oracle._lib = saved


CONTROLLER_MUTANTS = {
    "ties_expire": ("i64_out[0] = (cost[0] < cost[1]) ? 1 : 0;",
                    "i64_out[0] = (cost[0] <= cost[1]) ? 1 : 0;"),
    "branches_swapped": ("const double timers[2] = {t2, INFINITY};",
                         "const double timers[2] = {INFINITY, t2};"),
    "short_strict": ("if (W[i] <= tstar) n_short += 1;", "if (W[i] < tstar) n_short += 1;"),
    "count_strict": ("if (wait_s[i] <= t_star) c += 1;", "if (wait_s[i] < t_star) c += 1;"),
    "t_star_inverted": ("const double tstar = b3 / a1;", "const double tstar = a1 / b3;"),
    "no_restore_price": ("cost[k] = b2 * (double)restored[k] + b3 * (double)(total - restored[k]);",
                         "cost[k] = b3 * (double)(total - restored[k]);"),
}


def _controller_pins_pass(mod):
    from tests import test_controller_pins as C
    try:
        for seed in range(8):
            for c2 in (1, 2, 3):
                C.test_controller_is_the_exact_two_branch_replay(mod, seed, c2)
        C.test_controller_at_or_below_lambda_crit_keeps_retain(mod, 0.5)
        C.test_crossover_counts_the_break_even_wait(mod)
        for family in ("lognormal", "mixture"):
            C.test_controller_freezes_table6_branch(mod, family)
    except AssertionError:
        return False
    return True


def test_unmutated_controller_passes(oracle_mod):
    assert _controller_pins_pass(oracle_mod)


@pytest.mark.parametrize("name", sorted(CONTROLLER_MUTANTS))
def test_controller_mutant_is_caught(oracle_mod, tmp_path, name):
    old, new = CONTROLLER_MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    mpath = tmp_path / "mutant.c"
    mpath.write_text(src.replace(old, new))
    lib = tmp_path / "libmutant.so"
    oracle.compile_library(str(mpath), str(lib))
    saved = oracle._lib
    try:
        oracle._lib = oracle._configure(ctypes.CDLL(str(lib)))
        assert _controller_pins_pass(oracle) is False, f"mutant {name} survived"
    finally:
        oracle._lib = saved
