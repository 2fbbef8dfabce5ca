"""float64 oracle of the paper's training loss (test infrastructure).

Only the test suite, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg may use it; it shares nothing with the GPU library.

* Readout (Sec. 3.3 and App. C): a leaky integrator (LI) per class, with the
  LIF neuron's V/I dynamics and no spikes, driven by the last hidden layer's
  merged spike queue.  Its logit is the exponentially weighted integral of
  V over [0, tau_max] (Eq. weighted_leaky_integrator_full), taken interval by
  interval between input events with the closed form of Eq.
  weighted_leaky_integrator; tau_li = inf gives the unweighted integral of
  Eq. leaky_integrator.  The logits are scaled by a fixed temperature
  multiplier before the softmax cross-entropy (App. C, the option the paper
  keeps).
* Spike-count regularisers (App. E.1, Eq. loss): per neuron and sample, the
  maximum of V over each input interval from the interval's true start
  state (resets of earlier intervals applied, none inside the interval), the
  under- and over-firing hinge terms, their batch averages gated by the
  mean spike count against the target, and the individual over-firing term.

The exponent of Eq. weighted_leaky_integrator is regrouped: e^{t_i/tau_m}
e^{-t_i/T_m} = e^{-t_i/tau_li} (since 1/T_m = 1/tau_li + 1/tau_m), which keeps
every factor below 1 (the product as printed overflows float32 for t_i
beyond about 1.8 s at tau_m = 20 ms).
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np


@dataclass
class LiParams:
    tau_mem: float = 0.02       # tau_m of the readout neurons (s)
    tau_syn: float = 0.005      # tau_s (s)
    tau_li: float = 0.5         # weighting time constant tau_LI (s); inf: unweighted
    tau_max: float = 1.0        # end of the integration window (s)
    beta: float = 0.05          # logit temperature multiplier


def _tt(tau_li, tau):
    """T = tau_li tau / (tau_li + tau) (tau itself when tau_li is infinite)."""
    return tau if math.isinf(tau_li) else tau_li * tau / (tau_li + tau)


def li_interval_integral(q: LiParams, V, I, t0, t1):
    """Integral of e^{-t/tau_li} V(t) over [t0, t1] for the LI state (V, I)
    at t0 (Eq. weighted_leaky_integrator with the regrouped exponent; with
    tau_li = inf, Eq. leaky_integrator).  V, I may be arrays (classes)."""
    tm, ts = q.tau_mem, q.tau_syn
    gamma = I * ts / (tm - ts)
    Tm, Ts = _tt(q.tau_li, tm), _tt(q.tau_li, ts)
    w0 = 1.0 if math.isinf(q.tau_li) else math.exp(-t0 / q.tau_li)
    d = t1 - t0
    return (V + gamma) * w0 * Tm * (1.0 - math.exp(-d / Tm)) - gamma * w0 * Ts * (1.0 - math.exp(-d / Ts))


def li_readout(ev_t, ev_src, ev_n, WT, q: LiParams):
    """Logits z [B, N_cls] (before the temperature): per sample, walk the
    sorted queue; between consecutive events (and from the last event to
    tau_max) add the interval integral, then advance (V, I) to the next
    event with Eq. mem_pot and add the event's weights to I.  Events at or
    after tau_max do not contribute."""
    ev_t = np.asarray(ev_t, np.float64)
    ev_src = np.asarray(ev_src)
    WT = np.asarray(WT, np.float64)
    B = ev_t.shape[0]
    ncls = WT.shape[1]
    tm, ts = q.tau_mem, q.tau_syn
    ka = ts / (tm - ts)
    z = np.zeros((B, ncls))
    for b in range(B):
        V = np.zeros(ncls)
        I = np.zeros(ncls)
        t = 0.0
        for k in range(int(ev_n[b])):
            tk = ev_t[b, k]
            if tk >= q.tau_max:
                break
            z[b] += li_interval_integral(q, V, I, t, tk)
            d = tk - t
            em, es = math.exp(-d / tm), math.exp(-d / ts)
            V = V * em + ka * I * (em - es)
            I = I * es + WT[int(ev_src[b, k])]
            t = tk
        z[b] += li_interval_integral(q, V, I, t, q.tau_max)
    return z


def ce_with_temperature(z, labels, beta: float):
    """Mean softmax cross-entropy of beta * z against labels, and dL/dz."""
    y = beta * np.asarray(z, np.float64)
    y = y - y.max(axis=1, keepdims=True)
    p = np.exp(y)
    p /= p.sum(axis=1, keepdims=True)
    B = y.shape[0]
    loss = -np.mean(np.log(p[np.arange(B), labels]))
    onehot = np.zeros_like(p)
    onehot[np.arange(B), labels] = 1.0
    return float(loss), beta * (p - onehot) / B


def li_event_kernel(q: LiParams, t0):
    """Logit of one unit-weight event at t0 (the readout is linear in the
    weights, so z = sum_e W[src_e] G(t_e)), and dG/dt0: the integral of
    e^{-t/tau_li} kappa (e^{-(t-t0)/tau_m} - e^{-(t-t0)/tau_s}) over
    [t0, tau_max].  Used for the readout's gradients."""
    tm, ts = q.tau_mem, q.tau_syn
    ka = ts / (tm - ts)
    if t0 >= q.tau_max:
        return 0.0, 0.0
    Tm, Ts = _tt(q.tau_li, tm), _tt(q.tau_li, ts)
    w0 = 1.0 if math.isinf(q.tau_li) else math.exp(-t0 / q.tau_li)
    r = q.tau_max - t0
    am, as_ = math.exp(-r / Tm), math.exp(-r / Ts)
    G = ka * w0 * (Tm * (1.0 - am) - Ts * (1.0 - as_))
    inv_li = 0.0 if math.isinf(q.tau_li) else 1.0 / q.tau_li
    dG = -G * inv_li + ka * w0 * (as_ - am)
    return G, dG


def li_readout_grad(ev_t, ev_src, ev_n, WT, q: LiParams, dz):
    """Gradients of a loss with dL/dz = dz through the readout: dL/dW^T
    [C_in, N_cls] and dL/d(event time) [B, E_max] (0 on padding and at or
    after tau_max)."""
    ev_t = np.asarray(ev_t, np.float64)
    WT = np.asarray(WT, np.float64)
    B, E = ev_t.shape
    gW = np.zeros_like(WT)
    gt = np.zeros((B, E))
    for b in range(B):
        for k in range(int(ev_n[b])):
            G, dG = li_event_kernel(q, ev_t[b, k])
            c = int(ev_src[b, k])
            gW[c] += G * dz[b]
            gt[b, k] = dG * float(np.dot(WT[c], dz[b]))
    return gW, gt


# ---------------------------------------------------------------------------
# Spike-count regularisers (App. E.1)
# ---------------------------------------------------------------------------

@dataclass
class RegParams:
    c_target: float = 4.0        # target spike count per sample
    lam_reg: float = 1.0         # lambda_reg
    lam_over: float = 1.0        # lambda_over-reg


def interval_vmax(tm, ts, V0, I0, L):
    """Largest V over [0, L] of the no-reset trajectory from (V0, I0) (Eq.
    t_vmax: the stationary point where it lies inside, else the larger end;
    L = inf allowed).  Also returns the time u of the maximum."""
    ka = ts / (tm - ts)
    best, ub = V0, 0.0
    if not math.isinf(L):
        em, es = math.exp(-L / tm), math.exp(-L / ts)
        V1 = V0 * em + ka * I0 * (em - es)
        if V1 > best:
            best, ub = V1, L
    # dV/du = 0: (V0 + ka I0)/tm e^{-u/tm} = ka I0/ts e^{-u/ts}
    if I0 > 0.0 and V0 + ka * I0 > 0.0:
        ratio = ka * I0 * tm / ((V0 + ka * I0) * ts)
        if ratio > 1.0:
            u = math.log(ratio) * tm * ts / (tm - ts)
            if 0.0 < u < L:
                em, es = math.exp(-u / tm), math.exp(-u / ts)
                Vu = V0 * em + ka * I0 * (em - es)
                if Vu > best:
                    best, ub = Vu, u
    return best, ub


def interval_table(ev_t, n, WT_col, out_t, out_k, ns, tm, ts, th, vr, t_end):
    """Per input interval j = 0 .. n of one (sample, neuron): the interval
    (t_{j-1}, t_j] (t_{-1} = 0; j = n is the open interval up to t_end), the
    true (V, I) at its start (resets of the spikes of earlier intervals
    applied), its V_max (interval_vmax, no reset inside), the time of that
    maximum, and whether a spike lies in it (out_k[s] == j)."""
    ka = ts / (tm - ts)
    rows = []
    spiked = np.zeros(n + 1, bool)
    for s in range(ns):
        spiked[int(out_k[s])] = True
    V, I, t = 0.0, 0.0, 0.0
    s = 0
    for j in range(n + 1):
        t1 = float(ev_t[j]) if j < n else t_end
        L = t1 - t
        vmax, u = interval_vmax(tm, ts, V, I, L)
        rows.append((t, t1, V, I, vmax, u, bool(spiked[j])))
        # advance to the interval's end with its spikes (hard reset to vr)
        while s < ns and int(out_k[s]) == j:
            d = float(out_t[s]) - t
            em, es = math.exp(-d / tm), math.exp(-d / ts)
            I = I * es
            V = vr
            t = float(out_t[s])
            s += 1
        if j < n:
            d = t1 - t
            em, es = math.exp(-d / tm), math.exp(-d / ts)
            V = V * em + ka * I * (em - es)
            I = I * es + float(WT_col[j])
            t = t1
    return rows


def spike_count_reg(tables, counts, th, rp: RegParams):
    """L_reg and L_over-reg (App. E.1) from the interval tables of every
    (sample, neuron) of a layer: tables[b][i] = interval_table rows, counts
    [B, N] spike counts.  Empty interval sets give a zero term.  Returns
    (L_reg, L_over, dL/dV_max as a list per (b, i) of per-interval
    coefficients) for L = lam_reg L_reg + lam_over L_over, taking the gating
    factors (functions of the counts) as constants."""
    B, N = counts.shape
    under = np.zeros((B, N))
    over = np.zeros((B, N))
    for b in range(B):
        for i in range(N):
            rows = tables[b][i]
            sil = [r[4] for r in rows if not r[6]]
            spk = [r[4] for r in rows if r[6]]
            under[b, i] = np.mean([max(th - v, 0.0) for v in sil]) if sil else 0.0
            over[b, i] = np.mean([max(v - th, 0.0) for v in spk]) if spk else 0.0
    cbar = counts.mean(axis=0)
    gu = np.maximum(1.0 - cbar / rp.c_target, 0.0)
    go = np.maximum(cbar / rp.c_target - 1.0, 0.0)
    L_reg = float(np.mean(gu * under.mean(axis=0) + go * over.mean(axis=0)))
    gi = np.maximum(counts / rp.c_target - 1.0, 0.0)
    L_over = float((gi * over).sum() / N)
    coef = []
    for b in range(B):
        row = []
        for i in range(N):
            rows = tables[b][i]
            nsil = sum(1 for r in rows if not r[6])
            nspk = sum(1 for r in rows if r[6])
            cs = []
            for r in rows:
                v = r[4]
                if r[6]:
                    a = (rp.lam_reg * go[i] / (N * B) + rp.lam_over * gi[b, i] / N) / nspk
                    cs.append(a if v > th else 0.0)
                else:
                    a = rp.lam_reg * gu[i] / (N * B) / nsil
                    cs.append(-a if v < th else 0.0)
            row.append(cs)
        coef.append(row)
    return L_reg, L_over, coef


def spike_count_reg_grad(ev_t, ev_src, ev_n, WT, out_t, out_k, out_n, tm, ts, th, vr, t_end, rp: RegParams):
    """Gradient of lam_reg L_reg + lam_over L_over (App. E.1, Eq. loss) with
    the gates held constant (they are functions of the spike counts, which are
    piecewise constant in the parameters).  Each V_max is the value of the
    interval's trajectory at its argmax tau = t0 + u:
        V(tau) = sum_{k < j} w_k K(tau - t_k) - (th - vr) sum_{s: out_k < j} e^{-(tau - t_s)/tm},
    with K(u) = kappa (e^{-u/tm} - e^{-u/ts}).  Its derivative takes the
    explicit dependence on the weights, the input times and the spike times
    before the interval, plus V'(tau) times the motion of tau when the argmax
    is an interval end that is an input time (zero at an interior maximum,
    where V' = 0).  Returns (L_reg, L_over, gW_direct [C, N], gT_direct
    [B, E_max], g_spike [B, N, s_max]); the full gradient adds the layer's
    backward pass (App. D.3) of the upstream spike-time gradient g_spike."""
    B, N = out_n.shape
    C = WT.shape[0]
    E = ev_t.shape[1]
    S = out_t.shape[2]
    ka = ts / (tm - ts)
    tables = []
    for b in range(B):
        n = int(ev_n[b])
        row = []
        for i in range(N):
            ns = int(out_n[b, i])
            w = WT[ev_src[b, :n], i]
            row.append(interval_table(ev_t[b, :n], n, w, out_t[b, i, :ns], out_k[b, i, :ns], ns, tm, ts, th, vr, t_end))
        tables.append(row)
    L_reg, L_over, coef = spike_count_reg(tables, out_n, th, rp)
    gW = np.zeros((C, N))
    gT = np.zeros((B, E))
    gS = np.zeros((B, N, S))
    for b in range(B):
        n = int(ev_n[b])
        t = np.asarray(ev_t[b, :n], np.float64)
        src = np.asarray(ev_src[b, :n])
        for i in range(N):
            w = np.asarray(WT[src, i], np.float64)
            ns = int(out_n[b, i])
            st = np.asarray(out_t[b, i, :ns], np.float64)
            sk = np.asarray(out_k[b, i, :ns])
            for j, (t0, t1, V0, I0, vmax, u, spiked) in enumerate(tables[b][i]):
                c = coef[b][i][j]
                if c == 0.0:
                    continue
                tau = t0 + u
                # the input events before the interval (k < j)
                d = tau - t[:j]
                em, es = np.exp(-d / tm), np.exp(-d / ts)
                np.add.at(gW[:, i], src[:j], c * ka * (em - es))
                gT[b, :j] += -c * w[:j] * ka * (-em / tm + es / ts)
                # the spikes before the interval
                before = sk < j
                gS[b, i, :ns][before] += c * (-(th - vr) / tm) * np.exp(-(tau - st[before]) / tm)
                # an argmax at an interval end that is an input time moves with it
                L = t1 - t0
                if u == 0.0 and j > 0:
                    gT[b, j - 1] += c * (I0 - V0) / tm
                elif j < n and u == L and L > 0.0:
                    emL, esL = math.exp(-L / tm), math.exp(-L / ts)
                    V1 = V0 * emL + ka * I0 * (emL - esL)
                    gT[b, j] += c * (I0 * esL - V1) / tm
    return L_reg, L_over, gW, gT, gS


# ---------------------------------------------------------------------------
# The same regularisers on a layer with synaptic delays
# ---------------------------------------------------------------------------

def delayed_interval_tables(ev_src, ev_n, WT, q_t, q_k, out_t, out_k, out_n, tm, ts, th, vr, t_end):
    """interval_table of every (sample, neuron) of a layer with synaptic
    delays (Sec. 3.1 Eq. spike_input): a neuron's input sequence is its own
    arrival queue q_t[b, i], q_k[b, i] (App. E.2; oracle.delay_queues), so its
    intervals lie between consecutive arrivals and out_k counts queue events.
    Returns tables[b][i]."""
    B, N = out_n.shape
    tables = []
    for b in range(B):
        n = int(ev_n[b])
        row = []
        for i in range(N):
            ns = int(out_n[b, i])
            k = np.asarray(q_k[b, i, :n])
            w = WT[np.asarray(ev_src[b])[k], i]
            row.append(interval_table(q_t[b, i, :n], n, w, out_t[b, i, :ns], out_k[b, i, :ns], ns, tm, ts, th, vr,
                                      t_end))
        tables.append(row)
    return tables


def spike_count_reg_delayed_grad(ev_t, ev_src, ev_n, WT, q_t, q_k, out_t, out_k, out_n, tm, ts, th, vr, t_end,
                                 rp: RegParams):
    """spike_count_reg_grad for a layer with synaptic delays: every input
    time of a neuron is its arrival a = t_k + d_{src_k, i} (its queue,
    q_t / q_k), so a term of dL/da goes both to dL/dt_k and to
    dL/dd_{src_k, i} (d a / d t_k = d a / d d = 1).  Returns (L_reg, L_over,
    gW_direct [C, N], gD_direct [C, N], gT_direct [B, E_max], g_spike
    [B, N, s_max])."""
    B, N = out_n.shape
    C = WT.shape[0]
    E = ev_t.shape[1]
    S = out_t.shape[2]
    ka = ts / (tm - ts)
    tables = delayed_interval_tables(ev_src, ev_n, WT, q_t, q_k, out_t, out_k, out_n, tm, ts, th, vr, t_end)
    L_reg, L_over, coef = spike_count_reg(tables, out_n, th, rp)
    gW = np.zeros((C, N))
    gD = np.zeros((C, N))
    gT = np.zeros((B, E))
    gS = np.zeros((B, N, S))
    for b in range(B):
        n = int(ev_n[b])
        for i in range(N):
            k = np.asarray(q_k[b, i, :n], np.int64)
            a = np.asarray(q_t[b, i, :n], np.float64)
            src = np.asarray(ev_src[b], np.int64)[k]
            w = np.asarray(WT[src, i], np.float64)
            ns = int(out_n[b, i])
            st = np.asarray(out_t[b, i, :ns], np.float64)
            sk = np.asarray(out_k[b, i, :ns])
            ga = np.zeros(n)                       # dL/da of each queue event
            for j, (t0, t1, V0, I0, vmax, u, spiked) in enumerate(tables[b][i]):
                c = coef[b][i][j]
                if c == 0.0:
                    continue
                tau = t0 + u
                # the arrivals before the interval (queue events r < j)
                d = tau - a[:j]
                em, es = np.exp(-d / tm), np.exp(-d / ts)
                np.add.at(gW[:, i], src[:j], c * ka * (em - es))
                ga[:j] += -c * w[:j] * ka * (-em / tm + es / ts)
                # the spikes before the interval
                before = sk < j
                gS[b, i, :ns][before] += c * (-(th - vr) / tm) * np.exp(-(tau - st[before]) / tm)
                # an argmax at an interval end that is an arrival moves with it
                L = t1 - t0
                if u == 0.0 and j > 0:
                    ga[j - 1] += c * (I0 - V0) / tm
                elif j < n and u == L and L > 0.0:
                    emL, esL = math.exp(-L / tm), math.exp(-L / ts)
                    V1 = V0 * emL + ka * I0 * (emL - esL)
                    ga[j] += c * (I0 * esL - V1) / tm
            np.add.at(gT[b], k, ga)
            np.add.at(gD[:, i], src, ga)
    return L_reg, L_over, gW, gD, gT, gS
