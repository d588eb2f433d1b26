"""C-ABI checks that need no GPU: the library loads, exports exactly what
include/kvr.h declares, sizes workspaces, and rejects bad arguments with the
documented status codes before touching the device."""
import ctypes
import math
import os
import re
import subprocess

import numpy as np
import pytest

import paper_2608_30830_amd as kvr
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kvr.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(kvr.LIB_PATH):
        from paper_2608_30830_amd import build
        build.build()
    return kvr.load_library()


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kvr_[a-z0-9_]+)\s*\(", text)))


def test_exports_match_header(lib):
    declared = _declared()
    assert declared == sorted(kvr.EXPORTS)
    out = subprocess.run(["nm", "-D", "--defined-only", kvr.LIB_PATH], check=True,
                         capture_output=True, text=True).stdout
    exported = sorted(set(re.findall(r"\bT (kvr_[a-z0-9_]+)\b", out)))
    assert exported == declared


def test_status_strings(lib):
    for code in range(0, -9, -1):
        s = kvr.status_string(code)
        assert s and s != "unknown status"
    assert kvr.status_string(12345) == "unknown status"


def test_price_helper_matches_oracle(lib, oracle_mod):
    """The library's Appendix B helper and the oracle's, written separately,
    agree to the bit on every workload's platform constants."""
    for name in ("tiny-exp-1k", "weibull-1m"):
        wl = workloads.make(name) if name == "tiny-exp-1k" else None
        kvb = workloads.KV_128K if wl is not None else workloads.KV_320K
        pf = workloads.PLATFORM
        a = kvr.kvr_prices_from_platform(kvb, pf["hbm_usable_bytes"], pf["host_link_bytes_per_s"],
                                         pf["prefill_tokens_per_s"], pf["n_gpu"],
                                         pf["host_slots_c2"], pf["w_ref_s"])
        b = oracle_mod.prices_from_platform(kvb, pf["hbm_usable_bytes"],
                                            pf["host_link_bytes_per_s"],
                                            pf["prefill_tokens_per_s"], pf["n_gpu"],
                                            pf["host_slots_c2"], pf["w_ref_s"])
        assert (a.a1_per_token, a.b2_per_token, a.b3_per_token) == (b.a1, b.b2, b.b3)
    with pytest.raises(kvr.KvrError) as ei:
        kvr.kvr_prices_from_platform(0.0, 1, 1, 1)
    assert ei.value.code == kvr.KVR_E_PRICE
    with pytest.raises(kvr.KvrError):
        kvr.kvr_prices_from_platform(float("nan"), 1, 1, 1)
    assert lib.kvr_prices_from_platform(1, 1, 1, 1, 1, 1, 1, None) == kvr.KVR_E_NULL


def _prices():
    return kvr.kvr_prices_from_platform(131072, 250e9, 50e9, 20000.0)


FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: every call below fails on the host


def _cost_grid_rc(lib, grid, prices=None, n=100, method=kvr.KVR_BRUTE, perm=None, ws=None,
                  ws_bytes=0, cost=FAKE):
    prices = _prices() if prices is None else prices
    sz = ctypes.c_size_t(ws_bytes)
    return lib.kvr_cost_grid(FAKE, FAKE, n, ctypes.byref(prices), ctypes.byref(grid.c), method,
                             cost, perm, ws, ctypes.byref(sz), None), sz.value


def test_workspace_size_query(lib):
    g = kvr.PolicyGrid([0.0], [10.0, 100.0, math.inf], [0.1, 0.5])
    rc, need = _cost_grid_rc(lib, g)
    assert rc == kvr.KVR_OK and need > 256
    rc, need_s = _cost_grid_rc(lib, g, method=kvr.KVR_SORTED, n=1 << 20)
    assert rc == kvr.KVR_OK and need_s > 20 * (1 << 20)
    sz = ctypes.c_size_t(0)
    wl = workloads.make("tiny-exp-1k")
    g4 = kvr.PolicyGrid(np.geomspace(1, 3600, 64), list(np.geomspace(10, 86400, 256)) + [math.inf],
                        np.linspace(0.05, 1.0, 32))
    rc = lib.kvr_bootstrap(None, None, 65536, None, 4096, 65536, ctypes.byref(_prices()),
                           ctypes.byref(g4.c), None, None, None, None, ctypes.byref(sz), None)
    assert rc == kvr.KVR_OK
    # fused selection: two candidate slots per wave (257 waves per resample) x 32 loads,
    # no cost tensor; recompute-share sums for the 64 x 256 finite deadlines per resample
    cands = 4096 * 257 * 2 * 32 * 16
    r3 = 4096 * 64 * 256 * 8
    assert cands + r3 <= sz.value < cands + r3 + (64 << 20)
    del wl


BAD_GRIDS = [
    ([math.nan], [1.0], [0.1], kvr.KVR_E_GRID),
    ([-1.0], [1.0], [0.1], kvr.KVR_E_GRID),
    ([math.inf], [1.0], [0.1], kvr.KVR_E_GRID),
    ([2.0, 1.0], [1.0], [0.1], kvr.KVR_E_GRID),
    ([1.0, 1.0], [1.0], [0.1], kvr.KVR_E_GRID),
    ([0.0], [math.nan], [0.1], kvr.KVR_E_GRID),
    ([0.0], [0.0], [0.1], kvr.KVR_E_GRID),
    ([0.0], [-5.0], [0.1], kvr.KVR_E_GRID),
    ([0.0], [math.inf, 5.0], [0.1], kvr.KVR_E_GRID),
    ([0.0], [5.0, 5.0], [0.1], kvr.KVR_E_GRID),
    ([0.0], [5.0, math.inf, math.inf], [0.1], kvr.KVR_E_GRID),
    ([0.0], [5.0], [math.nan], kvr.KVR_E_GRID),
    ([0.0], [5.0], [-0.5], kvr.KVR_E_GRID),
    ([0.0], [5.0], [math.inf], kvr.KVR_E_GRID),
    ([], [5.0], [0.1], kvr.KVR_E_SIZE),
    ([0.0], [], [0.1], kvr.KVR_E_SIZE),
    ([0.0], [5.0], [], kvr.KVR_E_SIZE),
    ([0.0], [5.0], [0.1] * 4097, kvr.KVR_E_SIZE),
]


@pytest.mark.parametrize("case", range(len(BAD_GRIDS)))
def test_bad_grid_rejected(lib, case):
    t1, t2, lam, want = BAD_GRIDS[case]
    g = kvr.PolicyGrid(t1, t2, lam)
    if not t1 or not t2 or not lam:
        # an empty array still needs a non-NULL pointer for the size check to be reached
        g.c.t1 = g.c.t1 if t1 else ctypes.cast(FAKE, ctypes.POINTER(ctypes.c_double))
        g.c.t2 = g.c.t2 if t2 else ctypes.cast(FAKE, ctypes.POINTER(ctypes.c_double))
        g.c.lam = g.c.lam if lam else ctypes.cast(FAKE, ctypes.POINTER(ctypes.c_double))
    assert _cost_grid_rc(lib, g)[0] == want


def test_too_many_policies(lib):
    g = kvr.PolicyGrid([0.0, 1.0], [5.0], [0.1])
    g.c.n_t1 = 1 << 12
    g.c.n_t2 = 1 << 13
    assert _cost_grid_rc(lib, g)[0] == kvr.KVR_E_SIZE


@pytest.mark.parametrize("field", ["a1_per_token", "b2_per_token", "b3_per_token",
                                   "host_slots_c2", "w_ref_s"])
@pytest.mark.parametrize("value", [0.0, -1.0, math.nan, math.inf])
def test_bad_price_rejected(lib, field, value):
    p = _prices()
    setattr(p, field, value)
    g = kvr.PolicyGrid([0.0], [5.0], [0.1])
    assert _cost_grid_rc(lib, g, prices=p)[0] == kvr.KVR_E_PRICE


@pytest.mark.parametrize("value", [-1e-9, -math.inf, math.nan, math.inf])
def test_bad_offload_charge_rejected(lib, value):
    """The optional offload charge may be 0 or positive, never negative or
    non-finite."""
    p = _prices()
    p.offload_per_token = value
    g = kvr.PolicyGrid([0.0], [5.0], [0.1])
    assert _cost_grid_rc(lib, g, prices=p)[0] == kvr.KVR_E_PRICE


def test_offload_charge_field(lib):
    """The header's price struct and the binding's agree field by field; the
    platform helper leaves the offload copy uncharged unless asked, and then
    charges it at the restore's per-token time; a positive charge passes the
    grid entry points' checks."""
    text = open(HEADER).read()
    body = text[text.index("typedef struct {\n    double a1_per_token;"):]
    body = body[:body.index("} kvr_prices;")]
    assert re.findall(r"double ([a-z0-9_]+);", body) == [f[0] for f in kvr.kvr_prices._fields_]
    assert ctypes.sizeof(kvr.kvr_prices) == 48
    assert _prices().offload_per_token == 0.0
    p = kvr.kvr_prices_from_platform(131072, 250e9, 50e9, 20000.0, charge_offload=True)
    assert p.offload_per_token == p.b2_per_token > 0.0
    g = kvr.PolicyGrid([0.0, 4.0], [5.0, math.inf], [0.1])
    assert _cost_grid_rc(lib, g, prices=p)[0] == kvr.KVR_OK
    t2 = ctypes.c_double()
    assert lib.kvr_eq3_timer(ctypes.byref(p), 0.5, ctypes.byref(t2)) == kvr.KVR_OK
    q = _prices()
    assert lib.kvr_eq3_timer(ctypes.byref(q), 0.5, ctypes.byref(ctypes.c_double())) == kvr.KVR_OK


def test_method_and_size_errors(lib):
    g = kvr.PolicyGrid([0.0], [5.0, math.inf], [0.1])
    assert _cost_grid_rc(lib, g, method=7)[0] == kvr.KVR_E_METHOD
    assert _cost_grid_rc(lib, g, method=kvr.KVR_BRUTE, perm=FAKE)[0] == kvr.KVR_E_METHOD
    assert _cost_grid_rc(lib, g, n=0)[0] == kvr.KVR_E_SIZE
    assert _cost_grid_rc(lib, g, n=1 << 31)[0] == kvr.KVR_E_SIZE
    p = _prices()
    assert lib.kvr_cost_grid(FAKE, FAKE, 10, ctypes.byref(p), ctypes.byref(g.c), 0, FAKE, None,
                             None, None, None) == kvr.KVR_E_NULL
    assert lib.kvr_cost_grid(FAKE, FAKE, 10, None, ctypes.byref(g.c), 0, FAKE, None,
                             None, ctypes.byref(ctypes.c_size_t()), None) == kvr.KVR_E_NULL


def test_workspace_errors(lib):
    g = kvr.PolicyGrid([0.0], [5.0, math.inf], [0.1])
    rc, need = _cost_grid_rc(lib, g)
    assert rc == kvr.KVR_OK
    assert _cost_grid_rc(lib, g, ws=FAKE, ws_bytes=need - 1)[0] == kvr.KVR_E_WORKSPACE
    assert _cost_grid_rc(lib, g, ws=ctypes.c_void_p(0x1008), ws_bytes=need)[0] == kvr.KVR_E_WORKSPACE
    # a workspace with a NULL output is a NULL error, not a launch
    assert _cost_grid_rc(lib, g, ws=FAKE, ws_bytes=need, cost=None)[0] == kvr.KVR_E_NULL


def test_bootstrap_and_select_errors(lib):
    g = kvr.PolicyGrid([0.0], [5.0, math.inf], [0.1])
    p = _prices()
    sz = ctypes.c_size_t(0)

    def boot(n=10, R=2, m=10):
        return lib.kvr_bootstrap(FAKE, FAKE, n, FAKE, R, m, ctypes.byref(p), ctypes.byref(g.c),
                                 FAKE, FAKE, None, None, ctypes.byref(sz), None)

    assert boot(R=0) == kvr.KVR_E_SIZE
    assert boot(m=0) == kvr.KVR_E_SIZE
    assert boot(n=0) == kvr.KVR_E_SIZE
    assert boot(R=1 << 30, m=1 << 11) == kvr.KVR_E_SIZE
    assert boot() == kvr.KVR_OK and sz.value > 0
    # 2^26 one-draw rows of an 8,192-policy grid: 2^33 waves, more than a launch holds
    big = kvr.PolicyGrid(list(np.arange(32.0)), list(np.geomspace(1.0, 1e5, 256)), [0.5])
    assert lib.kvr_bootstrap(FAKE, FAKE, 10, FAKE, 1 << 26, 1, ctypes.byref(p),
                             ctypes.byref(big.c), FAKE, FAKE, None, None, ctypes.byref(sz),
                             None) == kvr.KVR_E_SIZE
    assert lib.kvr_bootstrap(FAKE, FAKE, 10, FAKE, 1 << 16, 1, ctypes.byref(p),
                             ctypes.byref(big.c), FAKE, FAKE, None, None, ctypes.byref(sz),
                             None) == kvr.KVR_OK
    sel = lib.kvr_select_policy
    assert sel(None, 1, 1, 1, 2, 1, FAKE, FAKE, None, None) == kvr.KVR_E_NULL
    assert sel(FAKE, 0, 1, 1, 2, 1, FAKE, FAKE, None, None) == kvr.KVR_E_SIZE
    assert sel(FAKE, 1, 0, 1, 2, 1, FAKE, FAKE, None, None) == kvr.KVR_E_SIZE
    assert sel(FAKE, 1, 1, 1, 2, 2, FAKE, FAKE, None, None) == kvr.KVR_E_GRID
    # batch x n_lam beyond int32, including products that would overflow int64
    assert sel(FAKE, 1 << 20, 4096, 1, 2, 1, FAKE, FAKE, None, None) == kvr.KVR_E_SIZE
    assert sel(FAKE, 1 << 62, 4096, 1, 2, 1, FAKE, FAKE, None, None) == kvr.KVR_E_SIZE
    assert lib.kvr_workspace_status(None, None) == kvr.KVR_E_NULL


def test_factored_bootstrap_host_errors(lib):
    """kvr_bootstrap_factored validates like kvr_bootstrap and sizes its own
    workspace: sort buffers for n, bounded prefix rows per batch of resamples."""
    g = kvr.PolicyGrid([0.0, 2.0], [5.0, math.inf], [0.1, 0.2, 0.3])
    p = _prices()
    sz = ctypes.c_size_t(0)

    def boot(n=1000, R=2, m=1000, grid=g, prices=p, ws=None, best=FAKE):
        return lib.kvr_bootstrap_factored(FAKE, FAKE, n, FAKE, R, m, ctypes.byref(prices),
                                          ctypes.byref(grid.c), best, FAKE, None, ws,
                                          ctypes.byref(sz), None)

    assert boot(R=0) == kvr.KVR_E_SIZE
    assert boot(m=0) == kvr.KVR_E_SIZE
    assert boot(n=0) == kvr.KVR_E_SIZE
    assert boot(n=(1 << 31) - 1) == kvr.KVR_E_SIZE
    assert boot(R=1 << 30, m=1 << 11) == kvr.KVR_E_SIZE
    bad = _prices()
    bad.a1_per_token = -1.0
    assert boot(prices=bad) == kvr.KVR_E_PRICE
    assert boot(grid=kvr.PolicyGrid([0.0], [math.inf, 5.0], [0.1])) == kvr.KVR_E_GRID
    assert boot() == kvr.KVR_OK
    small = sz.value
    # per resample one row of N and S at the query slots: at most one slot per
    # t1 and deadline (2 + 4 here), at most n + 1
    assert small > 2 * 6 * 16 + 1001 * 4
    wide = kvr.PolicyGrid([0.0], list(np.geomspace(1.0, 1e5, 3000)), [0.1])
    assert boot(grid=wide) == kvr.KVR_OK
    assert sz.value - small > 2 * 1001 * 16           # slots capped at n + 1 = 1001 per row
    assert boot(R=100000, m=65536, n=65536) == kvr.KVR_OK
    assert sz.value < (2 << 30) + (64 << 20)          # count and query rows batched under 2 GiB
    assert boot(R=100000, m=65536, n=65536, grid=wide) == kvr.KVR_OK
    assert sz.value < (2 << 30) + (64 << 20)
    boot()
    sz.value = 1
    assert boot(ws=FAKE) == kvr.KVR_E_WORKSPACE
    boot()
    assert boot(ws=FAKE, best=None) == kvr.KVR_E_NULL


def test_eq3_timer_matches_oracle(lib, oracle_mod):
    """The library's Eq. 3 timer and the oracle's agree bit for bit."""
    p = kvr.kvr_prices_from_platform(327680, 250e9, 50e9, 20000.0)
    for mult in (0.0, 0.5, 1.0, 1.0000001, 2.0, 3.0, 17.0):
        lam = mult * 425.0 / 1800.0
        got = kvr.kvr_eq3_timer(p, lam)
        want = oracle_mod.eq3_timer(lam, p.b2_per_token, p.b3_per_token, 425.0, 1800.0)
        assert got == want or (math.isinf(got) and math.isinf(want))
    with pytest.raises(kvr.KvrError) as ei:
        kvr.kvr_eq3_timer(p, math.nan)
    assert ei.value.code == kvr.KVR_E_GRID
    assert lib.kvr_eq3_timer(ctypes.byref(p), 0.5, None) == kvr.KVR_E_NULL


def test_capacity_replay_host_errors(lib):
    p = _prices()
    t2 = (ctypes.c_double * 2)(600.0, math.inf)
    sz = ctypes.c_size_t(0)

    def call(reps=4, n=100, prices=p, timers=t2, k=2, ws=None):
        return lib.kvr_capacity_replay(FAKE, FAKE, None, reps, n, ctypes.byref(prices), timers, k,
                                       FAKE, None, None, ws, ctypes.byref(sz), None)

    assert call() == kvr.KVR_OK and sz.value > 0
    assert call(n=8193) == kvr.KVR_E_SIZE
    assert call(n=0) == kvr.KVR_E_SIZE
    assert call(reps=0) == kvr.KVR_E_SIZE
    assert call(k=0) == kvr.KVR_E_SIZE
    bad = (ctypes.c_double * 2)(600.0, math.nan)
    assert call(timers=bad) == kvr.KVR_E_GRID
    neg = (ctypes.c_double * 2)(0.0, 1.0)
    assert call(timers=neg) == kvr.KVR_E_GRID
    frac = _prices()
    frac.host_slots_c2 = 425.5
    assert call(prices=frac) == kvr.KVR_E_PRICE
    charged = _prices()
    charged.offload_per_token = charged.b2_per_token   # the replay has no offload charge
    assert call(prices=charged) == kvr.KVR_E_METHOD
    sz.value = 1                                   # far below the size needed
    assert call(ws=FAKE) == kvr.KVR_E_WORKSPACE
    assert lib.kvr_capacity_replay(FAKE, FAKE, None, 4, 100, ctypes.byref(p), None, 2, FAKE,
                                   None, None, None, ctypes.byref(sz), None) == kvr.KVR_E_NULL


def test_controller_out_layout():
    """The device-written result struct is 15 eight-byte fields, no padding,
    in the order the header declares."""
    assert ctypes.sizeof(kvr.kvr_controller_out) == 120
    assert kvr.kvr_controller_out.t2_s.offset == 64
    assert kvr.kvr_controller_out.p_short.offset == 112
    text = open(HEADER).read()
    body = text[text.index("typedef struct {\n    int64_t branch;"):]
    body = body[:body.index("} kvr_controller_out;")]
    names = re.findall(r"(?:int64_t|double) ([a-z0-9_]+)", body)
    assert names == [f[0] for f in kvr.kvr_controller_out._fields_]


def test_controller_host_errors(lib):
    p = _prices()
    sz = ctypes.c_size_t(0)

    def call(reps=4, n=100, prices=p, lam=0.5, ws=None, out=FAKE):
        return lib.kvr_controller_select(FAKE, FAKE, None, reps, n, ctypes.byref(prices), lam,
                                         out, ws, ctypes.byref(sz), None)

    assert call() == kvr.KVR_OK and sz.value > 0
    small = sz.value
    assert call(reps=64) == kvr.KVR_OK and sz.value > small
    assert call(n=8193) == kvr.KVR_E_SIZE
    assert call(n=0) == kvr.KVR_E_SIZE
    assert call(reps=0) == kvr.KVR_E_SIZE
    assert call(reps=2 ** 30) == kvr.KVR_E_SIZE
    for lam in (math.nan, -1.0, math.inf):
        assert call(lam=lam) == kvr.KVR_E_GRID
    frac = _prices()
    frac.host_slots_c2 = 425.5
    assert call(prices=frac) == kvr.KVR_E_PRICE
    zero = _prices()
    zero.a1_per_token = 0.0
    assert call(prices=zero) == kvr.KVR_E_PRICE
    charged = _prices()
    charged.offload_per_token = 1e-6                   # the replay has no offload charge
    assert call(prices=charged) == kvr.KVR_E_METHOD
    assert lib.kvr_controller_select(FAKE, FAKE, None, 4, 100, None, 0.5, FAKE, None,
                                     ctypes.byref(sz), None) == kvr.KVR_E_NULL
    assert lib.kvr_controller_select(FAKE, FAKE, None, 4, 100, ctypes.byref(p), 0.5, FAKE, None,
                                     None, None) == kvr.KVR_E_NULL
    sz.value = 1                                   # far below the size needed
    assert call(ws=FAKE) == kvr.KVR_E_WORKSPACE
    call()
    assert call(ws=FAKE, out=None) == kvr.KVR_E_NULL


def test_crossover_statistic_host_errors(lib):
    p = _prices()
    sz = ctypes.c_size_t(0)

    def call(n=100, prices=p, ws=None, count=FAKE):
        return lib.kvr_crossover_statistic(FAKE, n, ctypes.byref(prices), count, None, ws,
                                           ctypes.byref(sz), None)

    assert call() == kvr.KVR_OK and sz.value > 0
    assert call(n=0) == kvr.KVR_E_SIZE
    assert call(n=2 ** 41) == kvr.KVR_E_SIZE
    bad = _prices()
    bad.b3_per_token = math.nan
    assert call(prices=bad) == kvr.KVR_E_PRICE
    need = sz.value
    sz.value = need - 1
    assert call(ws=FAKE) == kvr.KVR_E_WORKSPACE
    sz.value = need
    assert call(ws=FAKE, count=None) == kvr.KVR_E_NULL


def test_product_path_has_no_cpu_fallback():
    """The binding never imports the oracle and has no CPU arithmetic path."""
    src = open(os.path.join(ROOT, "paper_2608_30830_amd", "__init__.py")).read()
    assert "oracle" not in src
    assert "numpy" not in src


def _noalloc_rc(lib, grid, n, method=kvr.KVR_SORTED, prices=None, perm=None, cost=FAKE):
    pr = prices if prices is not None else _prices()
    return lib.kvr_cost_grid_noalloc(FAKE, FAKE, n, ctypes.byref(pr), ctypes.byref(grid.c),
                                     method, cost, perm, None, None)


def test_noalloc_rejects_on_the_host(lib):
    """kvr_cost_grid_noalloc: the checks of kvr_cost_grid, and a workspace that
    would not fit the static scratch is KVR_E_SIZE, all before any device
    work (FAKE pointers are never touched)."""
    g = kvr.PolicyGrid([0.0], [10.0, 100.0, math.inf], [0.1, 0.9])
    bad = _prices()
    bad.b3_per_token = -1.0
    assert _noalloc_rc(lib, g, 100, prices=bad) == kvr.KVR_E_PRICE
    assert _noalloc_rc(lib, g, 0) == kvr.KVR_E_SIZE
    assert _noalloc_rc(lib, g, 100, method=7) == kvr.KVR_E_METHOD
    assert _noalloc_rc(lib, g, 100, method=kvr.KVR_BRUTE, perm=FAKE) == kvr.KVR_E_METHOD
    assert _noalloc_rc(lib, g, 100, cost=None) == kvr.KVR_E_NULL
    assert lib.kvr_cost_grid_noalloc(FAKE, FAKE, 100, None, ctypes.byref(g.c), 0, FAKE, None,
                                     None, None) == kvr.KVR_E_NULL
    # the sorted path needs about 40 bytes per wait: 2^21 waits exceed 64 MiB
    need = ctypes.c_size_t(0)
    pr = _prices()
    for n in (1 << 21, (1 << 31) - 1):
        assert lib.kvr_cost_grid(None, None, n, ctypes.byref(pr), ctypes.byref(g.c),
                                 kvr.KVR_SORTED, None, None, None, ctypes.byref(need),
                                 None) == kvr.KVR_OK
        assert need.value > kvr.NOALLOC_SCRATCH_BYTES
        assert _noalloc_rc(lib, g, n) == kvr.KVR_E_SIZE
    # brute force with more waits than the deadline bins of 64 MiB can hold
    # (nine GPU-tier timers: the general plan, which keeps a bin per wait; a
    # grid of at most eight t1 timers needs no per-wait storage)
    g9 = kvr.PolicyGrid([0.0] + [float(2 ** i) for i in range(8)], [10.0, 100.0, math.inf],
                        [0.1, 0.9])
    assert _noalloc_rc(lib, g9, 1 << 24, method=kvr.KVR_BRUTE) == kvr.KVR_E_SIZE


def test_noalloc_scratch_size_matches_header(lib):
    text = open(HEADER).read()
    m = re.search(r"#define KVR_NOALLOC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == kvr.NOALLOC_SCRATCH_BYTES
