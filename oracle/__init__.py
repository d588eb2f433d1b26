"""TEST INFRASTRUCTURE — the CPU oracle for the calibration replay.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s cpu_baseline
leg may import this package.  It is a plain, slow reference written from the
paper (Eq. 1, Eq. 3, Section 3.4, Appendices B and D); it shares no code with
the HIP library and never imports it.

``kvr_oracle.c`` holds the double loop, the closed form, the stable order and
the selection; ``exact.py`` holds an exact rational event simulation used to
pin the double loop on tiny inputs.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kvr_oracle.c")
# KVR_ORACLE_LIBRARY names another build of the oracle (e.g. one compiled with
# sanitizers), loaded as it is, without rebuilding.
_LIB_OVERRIDE = os.environ.get("KVR_ORACLE_LIBRARY")
_LIB = os.path.join(_HERE, "_build", "liboracle.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (-O2, no FP contraction, no fast-math)."""
    os.makedirs(os.path.dirname(_LIB), exist_ok=True)
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        compile_library(_SRC, tmp)
        os.replace(tmp, _LIB)
    return _LIB


def _configure(lib):
    """Declare the C signatures on a loaded copy of the oracle library."""
    D, I32, I64 = ctypes.c_double, ctypes.c_int32, ctypes.c_int64
    P = ctypes.c_void_p
    lib.oracle_prices_from_platform.argtypes = [D, D, D, D, D, P, P, P]
    lib.oracle_lambda_crit.argtypes = [D, D]
    lib.oracle_lambda_crit.restype = D
    lib.oracle_congestion_prices.argtypes = [P, I32, D, D, D, P]
    lib.oracle_eq3_timer.argtypes = [D, D, D, D, D]
    lib.oracle_eq3_timer.restype = D
    lib.oracle_cost_grid.argtypes = [P, P, I64, P, I64, D, D, D, D, D, D,
                                     P, I32, P, I32, P, I32, P]
    lib.oracle_select.argtypes = [P, I64, I32, I32, I32, P, P, P, P]
    lib.oracle_stable_order.argtypes = [P, I64, P]
    lib.oracle_closed_form_grid.argtypes = [P, P, I64, P, P, I64, D, D, D, D, D, D,
                                            P, I32, P, I32, P, I32, P]
    lib.oracle_closed_form_bootstrap.argtypes = [P, P, I64, P, I64, I64, D, D, D,
                                                 D, D, D, P, I32, P, I32, P, I32,
                                                 P, P]
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
    lib.oracle_capacity_replay.argtypes = [P, P, P, I64, I64, D, D, D, P, P]
    lib.oracle_capacity_replay.restype = D
    lib.oracle_capacity_replay_batch.argtypes = [P, P, P, I64, I64, I64, P, I32, D, D, P, P]
    lib.oracle_controller_select.argtypes = [P, P, P, I64, I64, I64, D, D, D, D, D, P, P]
    lib.oracle_crossover_count.argtypes = [P, I64, D, D]
    lib.oracle_crossover_count.restype = I64
    return lib


def compile_library(src: str, out: str) -> None:
    subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math",
                           "-fopenmp", "-shared", "-fPIC", "-std=c11",
                           "-Wall", "-Wextra", "-o", out, src, "-lm"])


def _load():
    global _lib
    if _lib is None:
        if _LIB_OVERRIDE:
            _lib = _configure(ctypes.CDLL(_LIB_OVERRIDE))
        else:
            build()
            _lib = _configure(ctypes.CDLL(_LIB))
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


class Prices:
    """Per-token price vector plus host capacity and reference wait.  boff is
    the optional per-token charge for the device-to-host copy at offload (0:
    uncharged, the paper's model)."""

    def __init__(self, a1, b2, b3, c2=425.0, w_ref=1800.0, boff=0.0):
        self.a1, self.b2, self.b3 = float(a1), float(b2), float(b3)
        self.c2, self.w_ref, self.boff = float(c2), float(w_ref), float(boff)

    def tuple(self):
        return (self.a1, self.b2, self.b3, self.boff, self.c2, self.w_ref)

    def __repr__(self):
        return (f"Prices(a1={self.a1!r}, b2={self.b2!r}, b3={self.b3!r}, c2={self.c2!r}, "
                f"w_ref={self.w_ref!r}, boff={self.boff!r})")


def prices_from_platform(kv_bytes_per_token, hbm_usable_bytes, host_link_bytes_per_s,
                         prefill_tokens_per_s, n_gpu=1.0, host_slots_c2=425.0,
                         w_ref_s=1800.0, charge_offload=False) -> Prices:
    """Appendix B price vector, per token.  With charge_offload the offload
    copy is charged at the restore's per-token time (the host link has the
    same bandwidth each way)."""
    lib = _load()
    a1, b2, b3 = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    lib.oracle_prices_from_platform(float(kv_bytes_per_token), float(hbm_usable_bytes),
                                    float(host_link_bytes_per_s), float(prefill_tokens_per_s),
                                    float(n_gpu), ctypes.byref(a1), ctypes.byref(b2),
                                    ctypes.byref(b3))
    return Prices(a1.value, b2.value, b3.value, host_slots_c2, w_ref_s,
                  b2.value if charge_offload else 0.0)


def workload_prices(wl) -> Prices:
    pf = wl.platform
    return prices_from_platform(wl.kv_bytes_per_token, pf["hbm_usable_bytes"],
                                pf["host_link_bytes_per_s"], pf["prefill_tokens_per_s"],
                                pf["n_gpu"], pf["host_slots_c2"], pf["w_ref_s"])


def lambda_crit(c2: float, w_ref: float) -> float:
    return _load().oracle_lambda_crit(float(c2), float(w_ref))


def congestion_prices(lam, b3, c2, w_ref) -> np.ndarray:
    lam = _f64(lam)
    out = np.empty_like(lam)
    _load().oracle_congestion_prices(_p(lam), lam.size, float(b3), float(c2),
                                     float(w_ref), _p(out))
    return out


def eq3_timer(lam, b2, b3, c2, w_ref) -> float:
    return _load().oracle_eq3_timer(float(lam), float(b2), float(b3), float(c2),
                                    float(w_ref))


def cost_grid(wait_s, ctx, prices: Prices, t1, t2, lam, idx_row=None) -> np.ndarray:
    """Double loop; returns cost[n_lam, n_t1, n_t2] (mean GPU-s per request)."""
    w, T = _f64(wait_s), _i32(ctx)
    t1, t2, lam = _f64(t1), _f64(t2), _f64(lam)
    idx = None if idx_row is None else _i32(idx_row)
    m = w.size if idx is None else idx.size
    out = np.empty((lam.size, t1.size, t2.size), dtype=np.float64)
    _load().oracle_cost_grid(_p(w), _p(T), w.size, _p(idx), m, *prices.tuple(),
                             _p(t1), t1.size, _p(t2), t2.size, _p(lam), lam.size,
                             _p(out))
    return out


def select(cost, t2):
    """cost[..., n_lam, n_t1, n_t2] -> (best, best_cost, branch), each [..., n_lam]."""
    cost = _f64(cost)
    t2 = _f64(t2)
    *lead, L, K1, K2 = cost.shape
    batch = int(np.prod(lead)) if lead else 1
    best = np.empty(batch * L, dtype=np.int32)
    bc = np.empty(batch * L, dtype=np.float64)
    br = np.empty(batch * L, dtype=np.int32)
    _load().oracle_select(_p(cost), batch, L, K1, K2, _p(t2), _p(best), _p(bc), _p(br))
    shape = tuple(lead) + (L,)
    return best.reshape(shape), bc.reshape(shape), br.reshape(shape)


def stable_order(wait_s) -> np.ndarray:
    w = _f64(wait_s)
    perm = np.empty(w.size, dtype=np.int32)
    _load().oracle_stable_order(_p(w), w.size, _p(perm))
    return perm


def closed_form_grid(wait_s, ctx, prices: Prices, t1, t2, lam, idx_row=None,
                     perm=None) -> np.ndarray:
    w, T = _f64(wait_s), _i32(ctx)
    t1, t2, lam = _f64(t1), _f64(t2), _f64(lam)
    perm = stable_order(w) if perm is None else _i32(perm)
    idx = None if idx_row is None else _i32(idx_row)
    m = w.size if idx is None else idx.size
    out = np.empty((lam.size, t1.size, t2.size), dtype=np.float64)
    _load().oracle_closed_form_grid(_p(w), _p(T), w.size, _p(perm), _p(idx), m,
                                    *prices.tuple(), _p(t1), t1.size, _p(t2), t2.size,
                                    _p(lam), lam.size, _p(out))
    return out


def closed_form_bootstrap(wait_s, ctx, idx, prices: Prices, t1, t2, lam):
    """Closed-form selection for every row of idx[R, m]: (best, best_cost) [R, n_lam]."""
    w, T, idx = _f64(wait_s), _i32(ctx), _i32(idx)
    t1, t2, lam = _f64(t1), _f64(t2), _f64(lam)
    R, m = idx.shape
    best = np.empty((R, lam.size), dtype=np.int32)
    bc = np.empty((R, lam.size), dtype=np.float64)
    _load().oracle_closed_form_bootstrap(_p(w), _p(T), w.size, _p(idx), R, m,
                                         *prices.tuple(), _p(t1), t1.size, _p(t2),
                                         t2.size, _p(lam), lam.size, _p(best), _p(bc))
    return best, bc


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Thread count of the oracle's later parallel loops (for timing it)."""
    _load().oracle_set_num_threads(int(n))


def capacity_replay(arrival_s, wait_s, c2, t2, b2, b3, ctx=None):
    """Finite-capacity admission replay of one request sequence under one
    host timer: (mean cost per request, restored tokens, admitted requests)."""
    a, w = _f64(arrival_s), _f64(wait_s)
    T = None if ctx is None else _i32(ctx)
    rest, adm = ctypes.c_int64(), ctypes.c_int64()
    cost = _load().oracle_capacity_replay(_p(a), _p(w), _p(T), a.size, int(c2), float(t2),
                                          float(b2), float(b3), ctypes.byref(rest),
                                          ctypes.byref(adm))
    return cost, rest.value, adm.value


def capacity_replay_batch(arrival_s, wait_s, c2, t2, b2, b3, ctx=None):
    """Rows [reps, n] of arrivals and waits x timers t2[K] -> (cost, restored) [reps, K]."""
    a, w = _f64(arrival_s), _f64(wait_s)
    T = None if ctx is None else _i32(ctx)
    t2 = _f64(t2)
    reps, n = a.shape
    cost = np.empty((reps, t2.size), dtype=np.float64)
    rest = np.empty((reps, t2.size), dtype=np.int64)
    _load().oracle_capacity_replay_batch(_p(a), _p(w), _p(T), reps, n, int(c2), _p(t2), t2.size,
                                         float(b2), float(b3), _p(cost), _p(rest))
    return cost, rest


class Controller:
    """The frozen host branch and the figures it was chosen from; index 0 of
    each pair is the Eq. 3 timer branch, index 1 host-retain."""
    I64 = ("branch", "restored_timer", "restored_retain", "admitted_timer",
           "admitted_retain", "total_tokens", "n_short", "n_requests")
    F64 = ("t2_s", "total_cost_timer", "total_cost_retain", "cost_per_request_timer",
           "cost_per_request_retain", "t_star_s", "p_short")

    def __init__(self, i64, f64):
        for k, v in zip(self.I64, i64):
            setattr(self, k, int(v))
        for k, v in zip(self.F64, f64):
            setattr(self, k, float(v))

    def as_tuple(self):
        return tuple(getattr(self, k) for k in self.I64 + self.F64)


def controller_select(arrival_s, wait_s, c2, lam, a1, b2, b3, w_ref=1800.0, ctx=None):
    """Section 3.4 controller on a calibration sample of rows [reps, n]."""
    a, w = np.atleast_2d(_f64(arrival_s)), np.atleast_2d(_f64(wait_s))
    T = None if ctx is None else _i32(ctx)
    reps, n = a.shape
    i64 = np.zeros(8, dtype=np.int64)
    f64 = np.zeros(7, dtype=np.float64)
    _load().oracle_controller_select(_p(a), _p(w), _p(T), reps, n, int(c2), float(lam),
                                     float(a1), float(b2), float(b3), float(w_ref),
                                     _p(i64), _p(f64))
    return Controller(i64, f64)


def crossover_count(wait_s, a1, b3) -> int:
    """Number of waits w <= t* = b3 / a1 (Section 4.3)."""
    w = _f64(wait_s).ravel()
    return int(_load().oracle_crossover_count(_p(w), w.size, float(a1), float(b3)))
