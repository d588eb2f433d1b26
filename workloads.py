"""Seeded synthetic inputs for the calibration replay.

This module only draws numbers and lays out grids.  It holds none of the
method's arithmetic (no prices, no costs, no selection): both the CPU oracle
under ``oracle/`` and the HIP library take their inputs from here, and
neither side imports the other.

Five workloads are defined, by what they are:

``tiny-exp-1k``
    1,000 waits ~ Exponential(mean 1,800 s); every context 8,192 tokens;
    t1 = {0}; 64 host timers log-spaced 10 s .. 4 h plus infinity;
    loads {0.25, 0.5, 0.75, 1.0} suspended req/s; KV 128 KiB/token.
``mix-64k``
    65,536 waits from 70 % LogNormal(median 60 s, sigma 1.0) and
    30 % LogNormal(median 7,200 s, sigma 0.8); contexts uniform integers in
    [2,048, 32,768]; t1 = {0}; 256 host timers log-spaced 1 s .. 24 h plus
    infinity; 16 loads evenly spaced 0.1 .. 1.0; KV 128 KiB/token.
``boot-1024x64k``
    1,024 with-replacement resamples (int32 index rows) of the mix-64k set,
    same timers and loads.
``weibull-1m``
    1,048,576 waits ~ Weibull(shape 0.5, scale 1,800 s) truncated at
    86,400 s (inverse CDF of the truncated law); contexts
    LogNormal(median 16,384, sigma 0.7) rounded and clipped to
    [1,024, 131,072]; 1,024 host timers log-spaced 1 s .. 24 h plus
    infinity; 64 loads 0.05 .. 1.0; KV 320 KiB/token.
``twotier-4096x64k``
    4,096 resamples of the mix-64k set; 64 GPU-tier timers t1 log-spaced
    1 s .. 1 h x 256 host timers log-spaced 10 s .. 24 h plus infinity x
    32 loads 0.05 .. 1.0; KV 128 KiB/token.

The wait families stand in for the paper's synthetic approval-wait families
(Section 4.1) and the context sizes for the approval-gated prefix statistics
of Section 2; no dataset is read.

Platform constants (shared by all five): usable HBM 250e9 B, host link
50e9 B/s each way, recompute 20,000 prefill tokens/s, one GPU, host capacity
C2 = 425 contexts, reference wait W_ref = 1,800 s.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

NAMES = ("tiny-exp-1k", "mix-64k", "boot-1024x64k", "weibull-1m",
         "twotier-4096x64k")

# Raw platform constants: inputs to each side's own price derivation.
PLATFORM = dict(
    hbm_usable_bytes=250e9,
    host_link_bytes_per_s=50e9,
    prefill_tokens_per_s=20000.0,
    n_gpu=1.0,
    host_slots_c2=425.0,
    w_ref_s=1800.0,
)
KV_128K = 32 * 8 * 128 * 2 * 2      # 131,072 B/token (32 layers, 8 KV heads, fp16)
KV_320K = 80 * 8 * 128 * 2 * 2      # 327,680 B/token (80 layers, 8 KV heads, fp16)


@dataclasses.dataclass
class Workload:
    name: str
    wait_s: np.ndarray          # float64 [n]
    ctx_tokens: np.ndarray      # int32 [n]
    t1: np.ndarray              # float64 [K1], ascending, finite
    t2: np.ndarray              # float64 [K2], ascending, last may be +inf
    lam: np.ndarray             # float64 [L], suspended requests per second
    kv_bytes_per_token: float
    idx: Optional[np.ndarray] = None   # int32 [R, m] or None
    platform: dict = dataclasses.field(default_factory=lambda: dict(PLATFORM))

    @property
    def n(self) -> int:
        return int(self.wait_s.shape[0])

    @property
    def n_resamples(self) -> int:
        return 1 if self.idx is None else int(self.idx.shape[0])

    @property
    def m(self) -> int:
        return self.n if self.idx is None else int(self.idx.shape[1])

    @property
    def evaluations(self) -> int:
        return (self.n_resamples * self.m * self.t1.size * self.t2.size
                * self.lam.size)


def _streams(seed: int):
    ss = np.random.SeedSequence(seed)
    return [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(3)]


def _with_inf(x: np.ndarray) -> np.ndarray:
    return np.concatenate([np.asarray(x, dtype=np.float64), [np.inf]])


def mixture_waits(rng: np.random.Generator, n: int) -> np.ndarray:
    """70 % LogNormal(median 60 s, sigma 1.0) + 30 % LogNormal(median 7,200 s, sigma 0.8)."""
    short = rng.random(n) < 0.7
    z = rng.standard_normal(n)
    return np.where(short, 60.0 * np.exp(1.0 * z), 7200.0 * np.exp(0.8 * z))


def truncated_weibull_waits(rng: np.random.Generator, n: int,
                            shape: float = 0.5, scale: float = 1800.0,
                            cap: float = 86400.0) -> np.ndarray:
    """Inverse-CDF draw from Weibull(shape, scale) conditioned on W <= cap."""
    f_cap = -math.expm1(-(cap / scale) ** shape)
    u = rng.random(n) * f_cap
    return scale * (-np.log1p(-u)) ** (1.0 / shape)


def _mix64k_base():
    rw, rt, _ = _streams(1001)
    w = mixture_waits(rw, 65536)
    t = rt.integers(2048, 32768, size=65536, endpoint=True).astype(np.int32)
    return w, t


def make(name: str, resamples: Optional[int] = None) -> Workload:
    """Build a workload by name.  ``resamples`` truncates the bootstrap batch
    to its first rows (the rows are drawn in order, so a truncated batch is a
    prefix of the full one)."""
    if name == "tiny-exp-1k":
        rw, _, _ = _streams(1000)
        w = rw.exponential(1800.0, 1000)
        t = np.full(1000, 8192, dtype=np.int32)
        return Workload(name, w, t, np.array([0.0]),
                        _with_inf(np.geomspace(10.0, 14400.0, 64)),
                        np.array([0.25, 0.5, 0.75, 1.0]), float(KV_128K))
    if name == "mix-64k":
        w, t = _mix64k_base()
        return Workload(name, w, t, np.array([0.0]),
                        _with_inf(np.geomspace(1.0, 86400.0, 256)),
                        np.linspace(0.1, 1.0, 16), float(KV_128K))
    if name == "boot-1024x64k":
        w, t = _mix64k_base()
        _, _, rb = _streams(1002)
        r = 1024 if resamples is None else resamples
        idx = bootstrap_rows(rb, r, 65536, 65536)
        return Workload(name, w, t, np.array([0.0]),
                        _with_inf(np.geomspace(1.0, 86400.0, 256)),
                        np.linspace(0.1, 1.0, 16), float(KV_128K), idx=idx)
    if name == "weibull-1m":
        rw, rt, _ = _streams(1003)
        n = 1 << 20
        w = truncated_weibull_waits(rw, n)
        z = rt.standard_normal(n)
        t = np.clip(np.rint(16384.0 * np.exp(0.7 * z)), 1024, 131072).astype(np.int32)
        return Workload(name, w, t, np.array([0.0]),
                        _with_inf(np.geomspace(1.0, 86400.0, 1024)),
                        np.linspace(0.05, 1.0, 64), float(KV_320K))
    if name == "twotier-4096x64k":
        w, t = _mix64k_base()
        _, _, rb = _streams(1004)
        r = 4096 if resamples is None else resamples
        idx = bootstrap_rows(rb, r, 65536, 65536)
        return Workload(name, w, t, np.geomspace(1.0, 3600.0, 64),
                        _with_inf(np.geomspace(10.0, 86400.0, 256)),
                        np.linspace(0.05, 1.0, 32), float(KV_128K), idx=idx)
    raise KeyError(f"unknown workload {name!r}; known: {NAMES}")


def sort_scale_case(log2n: int) -> Workload:
    """A large single sample for the sorted path's scaling: 2^log2n waits from
    the weibull-1m law (truncated Weibull(0.5, 1,800 s)) and its context law,
    with a small policy grid (t1 = 0, 64 log-spaced host timers 1 s - 24 h
    plus infinity, 4 loads) so that the sort and the scans dominate."""
    rw, rt, _ = _streams(1100 + log2n)
    n = 1 << log2n
    w = truncated_weibull_waits(rw, n)
    z = rt.standard_normal(n)
    t = np.clip(np.rint(16384.0 * np.exp(0.7 * z)), 1024, 131072).astype(np.int32)
    return Workload(f"sort-scale-2^{log2n}", w, t, np.array([0.0]),
                    _with_inf(np.geomspace(1.0, 86400.0, 64)),
                    np.array([0.25, 0.5, 0.75, 1.0]), float(KV_320K))


FAMILIES = ("lognormal", "exponential", "mixture")


def family_waits(rng: np.random.Generator, family: str, n: int,
                 short_weight: float = 0.5) -> np.ndarray:
    """The approval-wait families of Section 4.1, each with mean 1,800 s:
    LogNormal(sigma 1); Exponential; 0.5 Exp(mean 60 s) + 0.5 LogNormal(sigma
    0.7, mean 3,540 s).  ``short_weight`` changes the mixture's share of short
    approvals; the long component's mean then keeps the overall mean at
    1,800 s (3,540 s at the default 0.5)."""
    if family == "lognormal":
        return rng.lognormal(math.log(1800.0) - 0.5, 1.0, n)
    if family == "exponential":
        return rng.exponential(1800.0, n)
    if family == "mixture":
        if not 0.0 <= short_weight < 1.0:
            raise ValueError("short_weight must be in [0, 1)")
        long_mean = (1800.0 - 60.0 * short_weight) / (1.0 - short_weight)
        short = rng.random(n) < short_weight
        return np.where(short, rng.exponential(60.0, n),
                        rng.lognormal(math.log(long_mean) - 0.5 * 0.7 * 0.7, 0.7, n))
    raise KeyError(family)


# Table 3 price vectors, per request of the Section 4 model (alpha_1 GPU-s/s,
# beta_2 GPU-s, beta_3 GPU-s), with the host tier fixed at C2 = 425.
PLATFORM_PRICES = {"h100-nvl": (0.0176, 0.02, 1.91),
                   "a100-sxm": (0.0232, 0.02, 2.61),
                   "l40s": (0.118, 0.02, 5.14)}


def cross_platform_case(n: int = 65536, seed: int = 1005) -> Workload:
    """The second workload: the three Section 4.1 wait families (mean 1,800 s)
    side by side as one base sample of 3n waits, one context token each, with
    one index row per family (row f selects samples f*n .. f*n + n - 1); 64
    GPU-tier timers ({0} and 63 log-spaced 0.1 s - 1,000 s), 255 log-spaced
    host timers 10 s - 24 h plus infinity, loads 0.5, 1, 2, 3 x lambda_crit.
    It is priced with each PLATFORM_PRICES vector in turn."""
    rw, _, _ = _streams(seed)
    w = np.concatenate([family_waits(rw, f, n) for f in FAMILIES])
    t = np.ones(3 * n, dtype=np.int32)
    idx = np.arange(3 * n, dtype=np.int32).reshape(3, n)
    lc = 425.0 / 1800.0
    return Workload(f"platforms-3x{n // 1024}k", w, t,
                    np.concatenate([[0.0], np.geomspace(0.1, 1000.0, 63)]),
                    _with_inf(np.geomspace(10.0, 86400.0, 255)),
                    np.array([0.5, 1.0, 2.0, 3.0]) * lc, 1.0, idx=idx)


@dataclasses.dataclass
class ReplayCase:
    family: str
    rate_per_s: float
    arrival_s: np.ndarray    # float64 [reps, n], ascending per row (Poisson arrivals)
    wait_s: np.ndarray       # float64 [reps, n]

    @property
    def reps(self) -> int:
        return int(self.arrival_s.shape[0])

    @property
    def n(self) -> int:
        return int(self.arrival_s.shape[1])


def replay_case(family: str, rate_per_s: float, reps: int, n: int = 4000,
                seed: int = 2000, short_weight: float = 0.5) -> ReplayCase:
    """``reps`` independent request sequences of ``n`` suspensions: Poisson
    arrivals at ``rate_per_s`` starting at time 0, waits from ``family``
    (``short_weight`` as in family_waits; it also seeds the mixture's draws
    when it is not the default)."""
    fam = FAMILIES.index(family)
    key = [seed, fam, int(round(rate_per_s * 1e9))]
    if short_weight != 0.5:
        key.append(int(round(short_weight * 1e6)))
    ss = np.random.SeedSequence(key)
    ra, rw = [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(2)]
    arr = np.cumsum(ra.exponential(1.0 / rate_per_s, (reps, n)), axis=1)
    w = np.stack([family_waits(rw, family, n, short_weight) for _ in range(reps)])
    return ReplayCase(family, rate_per_s, arr, w)


def bootstrap_rows(rng: np.random.Generator, rows: int, m: int, n: int) -> np.ndarray:
    """``rows`` x ``m`` with-replacement index rows into ``n`` samples, drawn
    row by row so that any prefix of rows is reproducible on its own."""
    out = np.empty((rows, m), dtype=np.int32)
    for r in range(rows):
        out[r] = rng.integers(0, n, size=m, dtype=np.int32)
    return out


def random_case(seed: int, n: int, k1: int, k2: int, n_lam: int,
                resamples: int = 0, m: Optional[int] = None,
                inf_last: bool = True, ties: bool = False,
                kv_bytes_per_token: float = float(KV_128K)) -> Workload:
    """A small random case for parity tests: ragged sizes, duplicated waits
    (``ties``), optional bootstrap rows and an optional infinite timer."""
    rng = np.random.Generator(np.random.PCG64(seed))
    w = mixture_waits(rng, n)
    if ties and n > 4:
        # exact duplicates, exact zeros and waits sitting on timer values
        w[rng.integers(0, n, n // 4)] = w[0]
        w[rng.integers(0, n, max(1, n // 16))] = 0.0
    t = rng.integers(1, 40000, size=n, dtype=np.int32)
    t1 = np.zeros(1) if k1 == 1 else np.concatenate(
        [[0.0], np.geomspace(1.0, 3600.0, k1 - 1)])
    nfin = k2 - 1 if inf_last else k2
    t2 = np.geomspace(5.0, 90000.0, nfin)
    if inf_last:
        t2 = _with_inf(t2)
    if ties and n > 4:
        # a few waits exactly on a deadline t1 + t2 and on a t1
        for j in range(min(4, n)):
            a = int(rng.integers(0, t1.size))
            k = int(rng.integers(0, nfin))
            w[j + 1] = t1[a] + t2[k]
        w[-1] = t1[-1]
    lam = np.sort(rng.uniform(0.05, 1.2, n_lam))
    lam[0] = 0.1  # one uncongested load (below C2/W_ref = 0.2361)
    idx = None
    if resamples:
        mm = n if m is None else m
        idx = rng.integers(0, n, size=(resamples, mm), dtype=np.int32)
    return Workload(f"random-{seed}", w, t, t1, t2, lam, kv_bytes_per_token,
                    idx=idx)
