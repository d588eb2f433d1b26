"""TEST INFRASTRUCTURE — exact rational event simulation of the replay.

Each calibration request is walked through its own timeline, event by event,
in ``fractions.Fraction`` arithmetic (every float input is converted exactly):

* suspension at time 0 with the KV in HBM (state 1), holding price
  T * a1 per second, no resume cost (Section 3.1, Eq. 1, beta_1 = 0);
* at t1, if the request has not resumed, the copy moves to host DRAM
  (state 2), holding price T * a2(lambda) per second, where
  a2 = max(0, lambda - C2/W_ref) * b3 / C2 (Section 3.3, Eq. 3); the move
  itself costs boff * T (zero in the paper's model, which leaves the copy
  uncharged; a positive boff is the optional offload charge);
* the one-shot host timer fires at the deadline e (Appendix D); e is the
  deadline the controller actually arms, the binary64 value of t1 + t2;
  if the request is still suspended the host copy is discarded (state 3,
  alpha_3 = 0);
* at resume (time w) the request pays the resume cost of its current state:
  0 in HBM, b2 * T from host, b3 * T after a discard.

The mean over the sample, the arg-min per load (exact ties to the larger
flat index) and nothing else are computed.  This is slow on purpose and is
only used on tiny inputs to pin the floating-point oracle.
"""
from __future__ import annotations

from fractions import Fraction
import math
from typing import List, Sequence


def _fr(x: float) -> Fraction:
    return Fraction(float(x))


def _request_cost(w: Fraction, T: int, t1: Fraction, e, a1: Fraction,
                  a2: Fraction, b2: Fraction, b3: Fraction,
                  boff: Fraction = Fraction(0)) -> Fraction:
    """Walk one request's timeline.  ``e`` is a Fraction or None (no timer)."""
    # events after suspension, in time order: offload at t1, expiry at e, resume at w
    events = [(t1, 1, "offload")]
    if e is not None:
        events.append((e, 2, "expire"))
    events.append((w, 0, "resume"))   # resume wins a tie with any timer event
    events.sort(key=lambda ev: (ev[0], ev[1]))
    state, since, total = "hbm", Fraction(0), Fraction(0)
    hold = {"hbm": a1 * T, "host": a2 * T, "gone": Fraction(0)}
    for when, _, kind in events:
        total += hold[state] * (when - since)
        since = when
        if kind == "resume":
            total += {"hbm": Fraction(0), "host": b2 * T, "gone": b3 * T}[state]
            return total
        if kind == "offload" and state == "hbm":
            state = "host"
            total += boff * T
        elif kind == "expire" and state == "host":
            state = "gone"
    raise AssertionError("unreachable: every request resumes")


def congestion_price(lam: float, b3: float, c2: float, w_ref: float) -> Fraction:
    p = _fr(lam) - _fr(c2) / _fr(w_ref)
    if p < 0:
        p = Fraction(0)
    return p * _fr(b3) / _fr(c2)


def cost_grid(wait_s: Sequence[float], ctx: Sequence[int], prices, t1: Sequence[float],
              t2: Sequence[float], lam: Sequence[float], idx_row=None) -> List[List[List[Fraction]]]:
    """Exact mean cost[l][a][k] as Fractions."""
    a1, b2, b3 = _fr(prices.a1), _fr(prices.b2), _fr(prices.b3)
    boff = _fr(getattr(prices, "boff", 0.0))
    rows = list(range(len(wait_s))) if idx_row is None else [int(i) for i in idx_row]
    m = len(rows)
    out = []
    for lv in lam:
        a2 = congestion_price(lv, prices.b3, prices.c2, prices.w_ref)
        per_a = []
        for ta in t1:
            t1f = _fr(ta)
            per_k = []
            for tk in t2:
                e = None if math.isinf(tk) else _fr(float(ta) + float(tk))
                tot = Fraction(0)
                for i in rows:
                    tot += _request_cost(_fr(wait_s[i]), int(ctx[i]), t1f, e, a1, a2, b2, b3,
                                         boff)
                per_k.append(tot / m)
            per_a.append(per_k)
        out.append(per_a)
    return out


def select(cost) -> List[int]:
    """Exact arg-min per load over f = a*K2 + k; ties go to the larger f."""
    best = []
    for per_a in cost:
        flat = [c for per_k in per_a for c in per_k]
        bi = 0
        for f in range(1, len(flat)):
            if flat[f] <= flat[bi]:
                bi = f
        best.append(bi)
    return best


def capacity_replay(arrival_s, wait_s, c2, t2, b2, b3, ctx=None):
    """The admission replay of Appendix D written out with an explicit list of
    resident departure times (quadratic, for tiny inputs): departures at or
    before an arrival free their slots first; admit if fewer than c2 remain;
    an admitted request is restored if its wait is within the host timer.
    Returns (exact mean cost as a Fraction, restored tokens, admitted)."""
    residents = []
    restored = admitted = total = 0
    for i, (a, w) in enumerate(zip(arrival_s, wait_s)):
        T = 1 if ctx is None else int(ctx[i])
        total += T
        residents = [d for d in residents if not d <= a]
        if len(residents) < c2:
            admitted += 1
            if w <= t2:
                restored += T
                residents.append(float(a) + float(w))
            else:
                residents.append(float(a) + float(t2))
    n = len(arrival_s)
    cost = (_fr(b2) * restored + _fr(b3) * (total - restored)) / n
    return cost, restored, admitted
