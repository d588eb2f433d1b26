"""Shared helpers for tests: stratified wait samples, fixture readers, and
comparison utilities.  Nothing here implements the method's arithmetic."""
from __future__ import annotations

import math
import os

import numpy as np
from scipy import special

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
EPS = 2.0 ** -53


def strata(n):
    return (np.arange(n, dtype=np.float64) + 0.5) / n


def stratified_exponential(n, mean):
    return -mean * np.log1p(-strata(n))


def lognormal_mu(mean, sigma):
    return math.log(mean) - 0.5 * sigma * sigma


def stratified_lognormal(n, mean, sigma):
    return np.exp(lognormal_mu(mean, sigma) + sigma * special.ndtri(strata(n)))


def stratified_mixture(n):
    """Section 4.1 mixture: 0.5 Exp(mean 60 s) + 0.5 LogNormal(sigma 0.7, mean 3,540 s)."""
    h = n // 2
    return np.concatenate([stratified_exponential(h, 60.0),
                           stratified_lognormal(n - h, 3540.0, 0.7)])


def survival(family, t):
    if family == "exponential":
        return math.exp(-t / 1800.0)
    if family == "lognormal":
        mu = lognormal_mu(1800.0, 1.0)
        return 0.5 * math.erfc((math.log(t) - mu) / math.sqrt(2.0))
    if family == "mixture":
        mu = lognormal_mu(3540.0, 0.7)
        return 0.5 * math.exp(-t / 60.0) + 0.25 * math.erfc(
            (math.log(t) - mu) / (0.7 * math.sqrt(2.0)))
    raise KeyError(family)


def stratified_family(family, n):
    if family == "exponential":
        return stratified_exponential(n, 1800.0)
    if family == "lognormal":
        return stratified_lognormal(n, 1800.0, 1.0)
    if family == "mixture":
        return stratified_mixture(n)
    raise KeyError(family)


def read_table(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            rows.append(line.split())
    return rows


def rel_err(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.maximum(np.abs(b), np.finfo(np.float64).tiny)
    return np.abs(a - b) / den


def near_tie_ok(cost_ref, best_a, best_b, rtol):
    """Where two selections differ, both picks must be within ``rtol`` of each
    other under the reference costs (a tie within rounding); returns the
    number of such differences, raising if any difference is a real one."""
    *lead, L, K1, K2 = cost_ref.shape
    flat = cost_ref.reshape(-1, L, K1 * K2)
    ba = np.asarray(best_a).reshape(-1, L)
    bb = np.asarray(best_b).reshape(-1, L)
    diffs = 0
    for r in range(flat.shape[0]):
        for l in range(L):
            if ba[r, l] != bb[r, l]:
                ca, cb = flat[r, l, ba[r, l]], flat[r, l, bb[r, l]]
                if abs(ca - cb) > rtol * abs(cb):
                    raise AssertionError(
                        f"selection differs at row {r} load {l}: {ba[r, l]} vs {bb[r, l]}, "
                        f"costs {ca!r} vs {cb!r}")
                diffs += 1
    return diffs


def min_runner_up_gap(cost):
    """Smallest relative gap between the best and the best *different-valued*
    policy per (row, load): structural ties (bit-equal costs) are skipped."""
    *lead, L, K1, K2 = cost.shape
    flat = np.sort(cost.reshape(-1, K1 * K2), axis=1)
    gaps = []
    for row in flat:
        b = row[0]
        higher = row[row > b]
        if higher.size:
            gaps.append((higher[0] - b) / abs(b) if b != 0 else np.inf)
    return min(gaps) if gaps else np.inf
