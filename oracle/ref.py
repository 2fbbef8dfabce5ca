"""Pure-Python float64 reference for tiny inputs (test infrastructure).

A second, deliberately different transcription of the same definitions as
``lif_oracle.c``: Python floats and ``math`` only, and the spike time found by
the bisection algorithm of Appendix D.2 (bracket [0, t_Vmax], halving on the
sign of R = V - V_th) run until the bracket cannot shrink, instead of Newton.
Used only to cross-check the C oracle on small cases.
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple


def membrane(V0: float, I0: float, t: float, tm: float, ts: float) -> float:
    """Eq. mem_pot (Appendix A)."""
    if math.isinf(t):
        return 0.0
    return V0 * math.exp(-t / tm) + I0 * ts / (tm - ts) * (math.exp(-t / tm) - math.exp(-t / ts))


def current(I0: float, t: float, ts: float) -> float:
    """Eq. curr (Appendix A)."""
    return 0.0 if math.isinf(t) else I0 * math.exp(-t / ts)


def t_vmax(V0: float, I0: float, tm: float, ts: float):
    """Eq. t_vmax (Appendix D.1), or None when V has no interior maximum."""
    D = V0 * (tm - ts) + I0 * ts
    if not (I0 > V0 and D > 0.0):
        return None
    return tm * ts / (tm - ts) * math.log(I0 * tm / D)


def spike_in_interval(V0: float, I0: float, length: float, tm: float, ts: float, th: float):
    """Sec. 3.2.2 rule.  Returns the right end of the root bracket, or None."""
    tv = t_vmax(V0, I0, tm, ts)
    if membrane(V0, I0, length, tm, ts) >= th:
        return tv if (tv is not None and tv < length) else length
    if tv is not None and tv < length and membrane(V0, I0, tv, tm, ts) >= th:
        return tv
    return None


def bisect_root(V0: float, I0: float, hi: float, tm: float, ts: float, th: float) -> float:
    """Appendix D.2 bisection, iterated until the midpoint stops moving;
    returns t_high (the bracket end that satisfies V >= V_th)."""
    lo = 0.0
    while True:
        mid = 0.5 * (lo + hi)
        if mid <= lo or mid >= hi:
            return hi
        if membrane(V0, I0, mid, tm, ts) - th >= 0.0:
            hi = mid
        else:
            lo = mid


def simulate(times: Sequence[float], weights: Sequence[float], tm=0.02, ts=0.005, th=1.0, vr=0.0,
             t_end=math.inf, s_max=64) -> List[Tuple[float, float]]:
    """One neuron receiving input events (times[k], weights[k]) in order.
    Returns the list of (spike time, I at spike)."""
    out = []
    t_cur, V, I, k = 0.0, 0.0, 0.0, 0
    n = len(times)
    while True:
        t_hi = float(times[k]) if k < n else t_end
        length = t_hi - t_cur
        if length > 0.0:
            hi = spike_in_interval(V, I, length, tm, ts, th)
            if hi is not None:
                tau = bisect_root(V, I, hi, tm, ts, th)
                Istar = current(I, tau, ts)
                out.append((t_cur + tau, Istar))
                if len(out) >= s_max:
                    return out
                V, I, t_cur = vr, Istar, t_cur + tau
                continue
        if k >= n:
            return out
        if length > 0.0:
            V, I = membrane(V, I, length, tm, ts), current(I, length, ts)
        I += float(weights[k])
        t_cur = t_hi
        k += 1
