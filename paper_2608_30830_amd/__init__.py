"""Python binding of libkvr (MI355X calibration replay): argument marshalling only.

Every entry point forwards to the C ABI declared in ``include/kvr.h`` with
the same name; PyTorch provides device memory and the current HIP stream.
All computation runs in the library's HIP kernels.  There is no CPU path: if
the library is not built, or no GPU is visible, the calls raise.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Sequence, Tuple

_PKG = os.path.dirname(os.path.abspath(__file__))
# KVR_LIBRARY names another build of the same library (e.g. one whose host
# code is compiled with sanitizers); by default the in-tree build is loaded.
LIB_PATH = os.environ.get("KVR_LIBRARY") or os.path.join(_PKG, "_build", "libkvr.so")

KVR_OK = 0
KVR_E_NULL = -1
KVR_E_SIZE = -2
KVR_E_GRID = -3
KVR_E_PRICE = -4
KVR_E_WORKSPACE = -5
KVR_E_DOMAIN = -6
KVR_E_HIP = -7
KVR_E_METHOD = -8
KVR_BRUTE = 0
KVR_SORTED = 1
KVR_RETAIN = 0
KVR_EXPIRE = 1

EXPORTS = ("kvr_prices_from_platform", "kvr_cost_grid", "kvr_cost_grid_noalloc",
           "kvr_select_policy", "kvr_bootstrap",
           "kvr_bootstrap_factored", "kvr_eq3_timer", "kvr_capacity_replay",
           "kvr_controller_select", "kvr_crossover_statistic", "kvr_workspace_status",
           "kvr_set_profile_events", "kvr_status_string")


class kvr_prices(ctypes.Structure):
    _fields_ = [("a1_per_token", ctypes.c_double), ("b2_per_token", ctypes.c_double),
                ("b3_per_token", ctypes.c_double), ("host_slots_c2", ctypes.c_double),
                ("w_ref_s", ctypes.c_double), ("offload_per_token", ctypes.c_double)]


class kvr_policy_grid(ctypes.Structure):
    _fields_ = [("t1", ctypes.POINTER(ctypes.c_double)), ("n_t1", ctypes.c_int32),
                ("t2", ctypes.POINTER(ctypes.c_double)), ("n_t2", ctypes.c_int32),
                ("lam", ctypes.POINTER(ctypes.c_double)), ("n_lam", ctypes.c_int32)]


class kvr_controller_out(ctypes.Structure):
    """Device-written result of kvr_controller_select; in each pair index 0 is
    the Eq. 3 timer branch, index 1 host-retain."""
    _fields_ = [("branch", ctypes.c_int64), ("restored_tokens", ctypes.c_int64 * 2),
                ("admitted", ctypes.c_int64 * 2), ("total_tokens", ctypes.c_int64),
                ("n_short", ctypes.c_int64), ("n_requests", ctypes.c_int64),
                ("t2_s", ctypes.c_double), ("total_cost", ctypes.c_double * 2),
                ("cost_per_request", ctypes.c_double * 2), ("t_star_s", ctypes.c_double),
                ("p_short", ctypes.c_double)]


class KvrError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {status_string(code)} (status {code})")


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libkvr.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"libkvr is not built ({path}); run __graft_entry__.build()")
    lib = ctypes.CDLL(path)
    P, I32, I64, D = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    SZ = ctypes.POINTER(ctypes.c_size_t)
    lib.kvr_prices_from_platform.argtypes = [D, D, D, D, D, D, D, ctypes.POINTER(kvr_prices)]
    lib.kvr_prices_from_platform.restype = ctypes.c_int
    lib.kvr_cost_grid.argtypes = [P, P, I64, ctypes.POINTER(kvr_prices),
                                  ctypes.POINTER(kvr_policy_grid), I32, P, P, P, SZ, P]
    lib.kvr_cost_grid.restype = ctypes.c_int
    lib.kvr_cost_grid_noalloc.argtypes = [P, P, I64, ctypes.POINTER(kvr_prices),
                                          ctypes.POINTER(kvr_policy_grid), I32, P, P, P, P]
    lib.kvr_cost_grid_noalloc.restype = ctypes.c_int
    lib.kvr_select_policy.argtypes = [P, I64, I32, I32, I32, I32, P, P, P, P]
    lib.kvr_select_policy.restype = ctypes.c_int
    lib.kvr_bootstrap.argtypes = [P, P, I64, P, I64, I64, ctypes.POINTER(kvr_prices),
                                  ctypes.POINTER(kvr_policy_grid), P, P, P, P, SZ, P]
    lib.kvr_bootstrap.restype = ctypes.c_int
    lib.kvr_bootstrap_factored.argtypes = lib.kvr_bootstrap.argtypes
    lib.kvr_bootstrap_factored.restype = ctypes.c_int
    lib.kvr_workspace_status.argtypes = [P, P]
    lib.kvr_workspace_status.restype = ctypes.c_int
    lib.kvr_eq3_timer.argtypes = [ctypes.POINTER(kvr_prices), D, ctypes.POINTER(ctypes.c_double)]
    lib.kvr_eq3_timer.restype = ctypes.c_int
    lib.kvr_capacity_replay.argtypes = [P, P, P, I64, I64, ctypes.POINTER(kvr_prices), P, I32,
                                        P, P, P, P, SZ, P]
    lib.kvr_capacity_replay.restype = ctypes.c_int
    lib.kvr_controller_select.argtypes = [P, P, P, I64, I64, ctypes.POINTER(kvr_prices), D, P,
                                          P, SZ, P]
    lib.kvr_controller_select.restype = ctypes.c_int
    lib.kvr_crossover_statistic.argtypes = [P, I64, ctypes.POINTER(kvr_prices), P, P, P, SZ, P]
    lib.kvr_crossover_statistic.restype = ctypes.c_int
    lib.kvr_set_profile_events.argtypes = [P, P]
    lib.kvr_set_profile_events.restype = ctypes.c_int
    lib.kvr_status_string.argtypes = [ctypes.c_int]
    lib.kvr_status_string.restype = ctypes.c_char_p
    _lib = lib
    return lib


def status_string(code: int) -> str:
    return load_library().kvr_status_string(int(code)).decode()


def _check(code: int, where: str) -> None:
    if code != KVR_OK:
        raise KvrError(code, where)


def kvr_prices_from_platform(kv_bytes_per_token: float, hbm_usable_bytes: float,
                             host_link_bytes_per_s: float, prefill_tokens_per_s: float,
                             n_gpu: float = 1.0, host_slots_c2: float = 425.0,
                             w_ref_s: float = 1800.0, charge_offload: bool = False) -> kvr_prices:
    """With charge_offload the device-to-host copy at offload is charged at
    the restore's per-token time (offload_per_token = b2_per_token)."""
    out = kvr_prices()
    _check(load_library().kvr_prices_from_platform(
        float(kv_bytes_per_token), float(hbm_usable_bytes), float(host_link_bytes_per_s),
        float(prefill_tokens_per_s), float(n_gpu), float(host_slots_c2), float(w_ref_s),
        ctypes.byref(out)), "kvr_prices_from_platform")
    if charge_offload:
        out.offload_per_token = out.b2_per_token
    return out


class PolicyGrid:
    """Host arrays of a policy grid, kept alive while the ctypes view is used."""

    def __init__(self, t1: Sequence[float], t2: Sequence[float], lam: Sequence[float]):
        self._t1 = (ctypes.c_double * len(t1))(*[float(x) for x in t1])
        self._t2 = (ctypes.c_double * len(t2))(*[float(x) for x in t2])
        self._lam = (ctypes.c_double * len(lam))(*[float(x) for x in lam])
        self.n_t1, self.n_t2, self.n_lam = len(t1), len(t2), len(lam)
        self.last_inf = 1 if (len(t2) and math.isinf(float(t2[-1]))) else 0
        self.c = kvr_policy_grid(ctypes.cast(self._t1, ctypes.POINTER(ctypes.c_double)), self.n_t1,
                                 ctypes.cast(self._t2, ctypes.POINTER(ctypes.c_double)), self.n_t2,
                                 ctypes.cast(self._lam, ctypes.POINTER(ctypes.c_double)), self.n_lam)


def _torch():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("libkvr needs a visible GPU (torch.cuda.is_available() is False)")
    return torch


def _stream_ptr(stream) -> ctypes.c_void_p:
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(int(s.cuda_stream))


def _ptr(t) -> Optional[int]:
    return None if t is None else ctypes.c_void_p(int(t.data_ptr()))


def _need(t, dtype, name):
    torch = _torch()
    if t.device.type != "cuda" or t.dtype != dtype or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous {dtype} CUDA tensor")


def _need_shape(t, shape, name):
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, not {tuple(t.shape)}")


def _on_stream(stream, *tensors) -> None:
    """Tie buffers allocated here to a caller's stream: torch's caching
    allocator then does not hand their memory out again before the work queued
    on that stream has finished (the wrappers return before it has)."""
    if stream is None:
        return
    for t in tensors:
        if t is not None:
            t.record_stream(stream)


def _workspace(nbytes: int, ws=None):
    torch = _torch()
    if ws is not None:
        _need(ws, torch.uint8, "workspace")
        if ws.numel() >= nbytes:
            return ws
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device="cuda")


class CostGridCall:
    """A prepared kvr_cost_grid call: workspace and outputs allocated once, so
    that ``launch()`` only enqueues the library's kernels (as a serving loop
    or a benchmark would call it)."""

    def __init__(self, wait_s, ctx_tokens, prices: kvr_prices, grid: PolicyGrid,
                 method: int = KVR_BRUTE, want_perm: bool = False):
        torch = _torch()
        _need(wait_s, torch.float64, "wait_s")
        _need(ctx_tokens, torch.int32, "ctx_tokens")
        _need_shape(ctx_tokens, wait_s.shape, "ctx_tokens")
        self.lib = load_library()
        self.wait_s, self.ctx, self.prices, self.grid, self.method = wait_s, ctx_tokens, prices, \
            grid, method
        self.n = wait_s.numel()
        need = ctypes.c_size_t(0)
        _check(self.lib.kvr_cost_grid(None, None, self.n, ctypes.byref(prices), ctypes.byref(grid.c),
                                      method, None, None, None, ctypes.byref(need), None),
               "kvr_cost_grid(size)")
        self.ws = _workspace(need.value)
        self.ws_bytes = ctypes.c_size_t(self.ws.numel())
        self.cost = torch.empty((grid.n_lam, grid.n_t1, grid.n_t2), dtype=torch.float64,
                                device="cuda")
        self.perm = torch.empty(self.n, dtype=torch.int32, device="cuda") if want_perm else None

    def launch(self, stream=None) -> None:
        _check(self.lib.kvr_cost_grid(_ptr(self.wait_s), _ptr(self.ctx), self.n,
                                      ctypes.byref(self.prices), ctypes.byref(self.grid.c),
                                      self.method, _ptr(self.cost), _ptr(self.perm), _ptr(self.ws),
                                      ctypes.byref(self.ws_bytes), _stream_ptr(stream)),
               "kvr_cost_grid")
        _on_stream(stream, self.ws, self.cost, self.perm)

    def status(self, stream=None) -> int:
        return self.lib.kvr_workspace_status(_ptr(self.ws), _stream_ptr(stream))


def kvr_cost_grid(wait_s, ctx_tokens, prices: kvr_prices, grid: PolicyGrid, method: int = KVR_BRUTE,
                  want_perm: bool = False, out=None, workspace=None, stream=None,
                  check: bool = True):
    """cost[n_lam, n_t1, n_t2] (and perm[n] for KVR_SORTED with want_perm)."""
    torch = _torch()
    lib = load_library()
    _need(wait_s, torch.float64, "wait_s")
    _need(ctx_tokens, torch.int32, "ctx_tokens")
    n = wait_s.numel()
    _need_shape(ctx_tokens, wait_s.shape, "ctx_tokens")
    need = ctypes.c_size_t(0)
    _check(lib.kvr_cost_grid(None, None, n, ctypes.byref(prices), ctypes.byref(grid.c), method,
                             None, None, None, ctypes.byref(need), None), "kvr_cost_grid(size)")
    ws = _workspace(need.value, workspace)
    if out is not None:
        _need(out, torch.float64, "out")
        _need_shape(out, (grid.n_lam, grid.n_t1, grid.n_t2), "out")
    cost = out if out is not None else torch.empty((grid.n_lam, grid.n_t1, grid.n_t2),
                                                   dtype=torch.float64, device="cuda")
    perm = torch.empty(n, dtype=torch.int32, device="cuda") if want_perm else None
    have = ctypes.c_size_t(ws.numel())
    st = _stream_ptr(stream)
    _check(lib.kvr_cost_grid(_ptr(wait_s), _ptr(ctx_tokens), n, ctypes.byref(prices),
                             ctypes.byref(grid.c), method, _ptr(cost), _ptr(perm), _ptr(ws),
                             ctypes.byref(have), st), "kvr_cost_grid")
    _on_stream(stream, ws, cost, perm)
    if check:
        _check(lib.kvr_workspace_status(_ptr(ws), st), "kvr_cost_grid(device)")
    return (cost, perm) if want_perm else cost


NOALLOC_SCRATCH_BYTES = 64 << 20   # KVR_NOALLOC_SCRATCH_BYTES


def kvr_cost_grid_noalloc(wait_s, ctx_tokens, prices: kvr_prices, grid: PolicyGrid,
                          method: int = KVR_BRUTE, cost=None, perm=None, status=None,
                          stream=None):
    """kvr_cost_grid with the library's static device scratch as workspace: the
    library allocates nothing.  ``cost`` ([n_lam, n_t1, n_t2] float64), ``perm``
    ([n] int32, KVR_SORTED only) and ``status`` ([1] int32: KVR_OK or
    KVR_E_DOMAIN once the stream reaches the end of the call) are caller tensors
    (allocated here when None); returns (cost, perm, status) without
    synchronising."""
    torch = _torch()
    _need(wait_s, torch.float64, "wait_s")
    _need(ctx_tokens, torch.int32, "ctx_tokens")
    n = wait_s.numel()
    _need_shape(ctx_tokens, wait_s.shape, "ctx_tokens")
    if cost is None:
        cost = torch.empty((grid.n_lam, grid.n_t1, grid.n_t2), dtype=torch.float64, device="cuda")
    _need(cost, torch.float64, "cost")
    _need_shape(cost, (grid.n_lam, grid.n_t1, grid.n_t2), "cost")
    if perm is not None:
        _need(perm, torch.int32, "perm")
        _need_shape(perm, (n,), "perm")
    if status is None:
        status = torch.empty(1, dtype=torch.int32, device="cuda")
    _need(status, torch.int32, "status")
    _need_shape(status, (1,), "status")
    _check(load_library().kvr_cost_grid_noalloc(_ptr(wait_s), _ptr(ctx_tokens), n,
                                                ctypes.byref(prices), ctypes.byref(grid.c),
                                                method, _ptr(cost), _ptr(perm), _ptr(status),
                                                _stream_ptr(stream)),
           "kvr_cost_grid_noalloc")
    _on_stream(stream, cost, perm, status)
    return cost, perm, status


def kvr_select_policy(cost, last_t2_is_inf: bool, stream=None) -> Tuple:
    """cost[..., n_lam, n_t1, n_t2] -> (best, best_cost, branch), each [..., n_lam]."""
    torch = _torch()
    _need(cost, torch.float64, "cost")
    *lead, L, K1, K2 = cost.shape
    batch = 1
    for d in lead:
        batch *= d
    best = torch.empty((batch, L), dtype=torch.int32, device="cuda")
    bc = torch.empty((batch, L), dtype=torch.float64, device="cuda")
    br = torch.empty((batch, L), dtype=torch.int32, device="cuda")
    _check(load_library().kvr_select_policy(_ptr(cost), batch, L, K1, K2, int(bool(last_t2_is_inf)),
                                            _ptr(best), _ptr(bc), _ptr(br), _stream_ptr(stream)),
           "kvr_select_policy")
    _on_stream(stream, best, bc, br)
    shape = tuple(lead) + (L,)
    return best.reshape(shape), bc.reshape(shape), br.reshape(shape)


class BootstrapCall:
    """A prepared kvr_bootstrap call (or kvr_bootstrap_factored with
    ``factored=True``): outputs and workspace allocated once, so that
    ``launch()`` only enqueues the library's kernels."""

    def __init__(self, wait_s, ctx_tokens, idx, prices: kvr_prices, grid: PolicyGrid,
                 want_cost: bool = False, factored: bool = False):
        torch = _torch()
        _need(wait_s, torch.float64, "wait_s")
        _need(ctx_tokens, torch.int32, "ctx_tokens")
        _need(idx, torch.int32, "idx")
        if idx.dim() != 2:
            raise ValueError("idx must be [n_resamples, m]")
        _need_shape(ctx_tokens, wait_s.shape, "ctx_tokens")
        self.lib = load_library()
        self.name = "kvr_bootstrap_factored" if factored else "kvr_bootstrap"
        self.fn = getattr(self.lib, self.name)
        self.wait_s, self.ctx, self.idx = wait_s, ctx_tokens, idx
        self.prices, self.grid = prices, grid
        self.n = wait_s.numel()
        self.R, self.m = idx.shape
        self.best = torch.empty((self.R, grid.n_lam), dtype=torch.int32, device="cuda")
        self.best_cost = torch.empty((self.R, grid.n_lam), dtype=torch.float64, device="cuda")
        self.cost = (torch.empty((self.R, grid.n_lam, grid.n_t1, grid.n_t2), dtype=torch.float64,
                                 device="cuda") if want_cost else None)
        need = ctypes.c_size_t(0)
        _check(self.fn(None, None, self.n, None, self.R, self.m, ctypes.byref(prices),
                       ctypes.byref(grid.c), None, None, _ptr(self.cost) if want_cost else None,
                       None, ctypes.byref(need), None), f"{self.name}(size)")
        self.ws = _workspace(need.value)
        self.ws_bytes = ctypes.c_size_t(self.ws.numel())

    def launch(self, stream=None) -> None:
        _check(self.fn(_ptr(self.wait_s), _ptr(self.ctx), self.n, _ptr(self.idx), self.R, self.m,
                       ctypes.byref(self.prices), ctypes.byref(self.grid.c), _ptr(self.best),
                       _ptr(self.best_cost), _ptr(self.cost), _ptr(self.ws),
                       ctypes.byref(self.ws_bytes), _stream_ptr(stream)), self.name)
        _on_stream(stream, self.ws, self.best, self.best_cost, self.cost)

    def status(self, stream=None) -> int:
        return self.lib.kvr_workspace_status(_ptr(self.ws), _stream_ptr(stream))


def kvr_bootstrap(wait_s, ctx_tokens, idx, prices: kvr_prices, grid: PolicyGrid,
                  want_cost: bool = False, stream=None, check: bool = True,
                  factored: bool = False):
    """(best[R, n_lam], best_cost[R, n_lam]) and, with want_cost, cost[R, n_lam, n_t1, n_t2];
    ``factored=True`` calls kvr_bootstrap_factored."""
    call = BootstrapCall(wait_s, ctx_tokens, idx, prices, grid, want_cost, factored)
    call.launch(stream)
    if check:
        _check(call.status(stream), "kvr_bootstrap(device)")
    if want_cost:
        return call.best, call.best_cost, call.cost
    return call.best, call.best_cost


def kvr_eq3_timer(prices: kvr_prices, lam: float) -> float:
    """Eq. 3 host timer t2(lambda) (inf at or below lambda_crit)."""
    out = ctypes.c_double()
    _check(load_library().kvr_eq3_timer(ctypes.byref(prices), float(lam), ctypes.byref(out)),
           "kvr_eq3_timer")
    return out.value


def kvr_capacity_replay(arrival_s, wait_s, prices: kvr_prices, t2: Sequence[float],
                        ctx_tokens=None, stream=None, check: bool = True):
    """Finite-capacity admission replay of rows [n_reps, n] under each timer:
    (cost, restored_tokens, admitted), each [n_reps, n_t2]."""
    torch = _torch()
    lib = load_library()
    _need(arrival_s, torch.float64, "arrival_s")
    _need(wait_s, torch.float64, "wait_s")
    if ctx_tokens is not None:
        _need(ctx_tokens, torch.int32, "ctx_tokens")
    if arrival_s.dim() != 2 or tuple(wait_s.shape) != tuple(arrival_s.shape):
        raise ValueError("arrival_s and wait_s must both be [n_reps, n]")
    if ctx_tokens is not None:
        _need_shape(ctx_tokens, arrival_s.shape, "ctx_tokens")
    reps, n = arrival_s.shape
    K = len(t2)
    t2c = (ctypes.c_double * K)(*[float(x) for x in t2])
    need = ctypes.c_size_t(0)
    _check(lib.kvr_capacity_replay(None, None, None, reps, n, ctypes.byref(prices), t2c, K, None,
                                   None, None, None, ctypes.byref(need), None),
           "kvr_capacity_replay(size)")
    ws = _workspace(need.value)
    cost = torch.empty((reps, K), dtype=torch.float64, device="cuda")
    rest = torch.empty((reps, K), dtype=torch.int64, device="cuda")
    adm = torch.empty((reps, K), dtype=torch.int64, device="cuda")
    have = ctypes.c_size_t(ws.numel())
    st = _stream_ptr(stream)
    _check(lib.kvr_capacity_replay(_ptr(arrival_s), _ptr(wait_s), _ptr(ctx_tokens), reps, n,
                                   ctypes.byref(prices), t2c, K, _ptr(cost), _ptr(rest),
                                   _ptr(adm), _ptr(ws), ctypes.byref(have), st),
           "kvr_capacity_replay")
    _on_stream(stream, ws, cost, rest, adm)
    if check:
        _check(lib.kvr_workspace_status(_ptr(ws), st), "kvr_capacity_replay(device)")
    return cost, rest, adm


class ControllerCall:
    """kvr_controller_select with its buffers allocated once: launch() only
    enqueues the library's kernels; result() copies the device struct back."""

    def __init__(self, arrival_s, wait_s, prices: kvr_prices, lam: float, ctx_tokens=None):
        torch = _torch()
        self.lib = load_library()
        _need(arrival_s, torch.float64, "arrival_s")
        _need(wait_s, torch.float64, "wait_s")
        if ctx_tokens is not None:
            _need(ctx_tokens, torch.int32, "ctx_tokens")
        if arrival_s.dim() != 2 or tuple(wait_s.shape) != tuple(arrival_s.shape):
            raise ValueError("arrival_s and wait_s must both be [n_reps, n]")
        if ctx_tokens is not None and tuple(ctx_tokens.shape) != tuple(arrival_s.shape):
            raise ValueError("ctx_tokens must be [n_reps, n]")
        self.args = (arrival_s, wait_s, ctx_tokens)
        self.reps, self.n = arrival_s.shape
        self.prices, self.lam = prices, float(lam)
        need = ctypes.c_size_t(0)
        _check(self.lib.kvr_controller_select(None, None, None, self.reps, self.n,
                                              ctypes.byref(prices), self.lam, None, None,
                                              ctypes.byref(need), None),
               "kvr_controller_select(size)")
        self.ws = _workspace(need.value)
        self.out = torch.empty(ctypes.sizeof(kvr_controller_out), dtype=torch.uint8,
                               device="cuda")

    def launch(self, stream=None) -> None:
        """Enqueue on ``stream`` (default: the current stream at this call)."""
        a, w, T = self.args
        have = ctypes.c_size_t(self.ws.numel())
        _check(self.lib.kvr_controller_select(_ptr(a), _ptr(w), _ptr(T), self.reps, self.n,
                                              ctypes.byref(self.prices), self.lam,
                                              _ptr(self.out), _ptr(self.ws), ctypes.byref(have),
                                              _stream_ptr(stream)),
               "kvr_controller_select")
        _on_stream(stream, self.ws, self.out)

    def result(self, stream=None) -> kvr_controller_out:
        _check(self.lib.kvr_workspace_status(_ptr(self.ws), _stream_ptr(stream)),
               "kvr_controller_select(device)")
        host = self.out.cpu()
        res = kvr_controller_out()
        ctypes.memmove(ctypes.byref(res), host.data_ptr(), ctypes.sizeof(res))
        return res


def kvr_controller_select(arrival_s, wait_s, prices: kvr_prices, lam: float, ctx_tokens=None,
                          stream=None) -> kvr_controller_out:
    """Section 3.4 controller on a calibration sample [n_reps, n]."""
    call = ControllerCall(arrival_s, wait_s, prices, lam, ctx_tokens)
    call.launch(stream)
    return call.result(stream)


def kvr_crossover_statistic(wait_s, prices: kvr_prices, stream=None, check: bool = True):
    """P(W <= t*) of a wait sample: (count, fraction), device tensors of one element."""
    torch = _torch()
    lib = load_library()
    _need(wait_s, torch.float64, "wait_s")
    n = wait_s.numel()
    need = ctypes.c_size_t(0)
    _check(lib.kvr_crossover_statistic(None, n, ctypes.byref(prices), None, None, None,
                                       ctypes.byref(need), None), "kvr_crossover_statistic(size)")
    ws = _workspace(need.value)
    count = torch.empty(1, dtype=torch.int64, device="cuda")
    frac = torch.empty(1, dtype=torch.float64, device="cuda")
    have = ctypes.c_size_t(ws.numel())
    st = _stream_ptr(stream)
    _check(lib.kvr_crossover_statistic(_ptr(wait_s), n, ctypes.byref(prices), _ptr(count),
                                       _ptr(frac), _ptr(ws), ctypes.byref(have), st),
           "kvr_crossover_statistic")
    _on_stream(stream, ws, count, frac)
    if check:
        _check(lib.kvr_workspace_status(_ptr(ws), st), "kvr_crossover_statistic(device)")
    return count, frac


def kvr_set_profile_events(ev_begin, ev_end) -> None:
    """Record raw hipEvent_t handles (ints) around the main kernel of later
    calls from this thread; (None, None) stops."""
    b = None if ev_begin is None else ctypes.c_void_p(int(ev_begin))
    e = None if ev_end is None else ctypes.c_void_p(int(ev_end))
    _check(load_library().kvr_set_profile_events(b, e), "kvr_set_profile_events")


def kvr_workspace_status(ws, stream=None) -> int:
    return load_library().kvr_workspace_status(_ptr(ws), _stream_ptr(stream))
