"""Pins of the loss oracle (oracle/loss.py) against what the paper and the
mathematics fix: numerical quadrature of the readout integral, closed forms
of single events, finite differences, torch's cross-entropy, dense sampling
of the interval maximum, the superposition form of the reset dynamics, and
hand-computed regulariser values."""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import loss as OL
import workloads as W

TM, TS = 0.02, 0.005
KA = TS / (TM - TS)


def _v_superposed(t, times, w, tm=TM, ts=TS):
    """V(t) of a neuron without resets as a sum of unit responses."""
    u = t - np.asarray(times)
    m = u > 0
    return float(np.sum(np.asarray(w)[m] * KA * (np.exp(-u[m] / tm) - np.exp(-u[m] / ts))))


_XG, _WG = np.polynomial.legendre.leggauss(60)


def _gauss(f, a, b):
    """Integral of the smooth f over [a, b] by 60-point Gauss-Legendre (the
    integrands here are sums of exponentials within an interval)."""
    if b <= a:
        return 0.0
    s = 0.5 * (b - a) * _XG + 0.5 * (a + b)
    return 0.5 * (b - a) * float(np.sum(_WG * np.array([f(x) for x in s])))


def _case(seed, n=40, C=6, ncls=3, T=0.3):
    rng = np.random.default_rng(seed)
    t = np.sort(rng.random(n) * T).astype(np.float32)
    src = rng.integers(0, C, n).astype(np.int32)
    WT = rng.normal(0, 1.5, (C, ncls)).astype(np.float32)
    return t.reshape(1, -1), src.reshape(1, -1), np.array([n], np.int32), WT


@pytest.mark.parametrize("tau_li", [0.05, 0.5, math.inf])
def test_readout_matches_quadrature(tau_li):
    """Eq. weighted_leaky_integrator_full by Gauss-Legendre quadrature of
    the superposed V(t), interval by interval."""
    q = OL.LiParams(tau_li=tau_li, tau_max=0.35)
    t, src, n, WT = _case(1)
    z = OL.li_readout(t, src, n, WT, q)
    knots = [0.0] + [float(x) for x in t[0]] + [q.tau_max]
    for c in range(WT.shape[1]):
        w = WT[src[0], c].astype(np.float64)
        f = lambda s: (1.0 if math.isinf(tau_li) else math.exp(-s / tau_li)) * _v_superposed(s, t[0], w)
        ref = sum(_gauss(f, a, b) for a, b in zip(knots[:-1], knots[1:]))
        assert abs(z[0, c] - ref) <= 1e-13 * max(1.0, abs(ref)), (c, z[0, c], ref)


def test_readout_window_cuts_late_events_and_far_times():
    """Events at or after tau_max add nothing; late event times (t/tau_m
    far beyond the float32 range of e^{t/tau_m}) stay finite and match
    quadrature (the regrouped exponent)."""
    q = OL.LiParams(tau_li=1.0, tau_max=3.05)
    t = np.array([[2.9, 2.95, 3.0, 3.1]], np.float32)
    src = np.array([[0, 1, 0, 1]], np.int32)
    WT = np.array([[2.0], [-1.0]], np.float32)
    z = OL.li_readout(t, src, np.array([4], np.int32), WT, q)
    assert np.isfinite(z).all()
    w = WT[src[0, :3], 0].astype(np.float64)
    f = lambda s: math.exp(-s / q.tau_li) * _v_superposed(s, t[0, :3], w)
    knots = [float(x) for x in t[0, :3]] + [3.05]
    ref = sum(_gauss(f, a, b) for a, b in zip(knots[:-1], knots[1:]))
    assert abs(z[0, 0] - ref) <= 1e-12 * abs(ref)
    z3 = OL.li_readout(t[:, :3], src[:, :3], np.array([3], np.int32), WT, q)
    assert z3[0, 0] == z[0, 0]


def test_single_event_closed_forms():
    """One event of weight w at t0: the unweighted integral over [t0, inf)
    is w kappa (tau_m - tau_s) = w tau_s; the weighted one is the event
    kernel G(t0), which the interval walk reproduces."""
    q = OL.LiParams(tau_li=math.inf, tau_max=200.0)
    z = OL.li_readout(np.array([[0.1]], np.float32), np.array([[0]], np.int32), np.array([1], np.int32),
                      np.array([[3.0]], np.float32), q)
    assert abs(z[0, 0] - 3.0 * TS) < 1e-13
    q = OL.LiParams(tau_li=0.2, tau_max=0.4)
    for t0 in (0.0, 0.05, 0.3, 0.3999):
        z = OL.li_readout(np.array([[t0]], np.float32), np.array([[0]], np.int32), np.array([1], np.int32),
                          np.array([[1.0]], np.float32), q)
        G, _ = OL.li_event_kernel(q, float(np.float32(t0)))
        assert abs(z[0, 0] - G) <= 1e-14 + 1e-12 * abs(G)


def test_readout_gradients_match_finite_differences():
    q = OL.LiParams(tau_li=0.3, tau_max=0.3)
    t, src, n, WT = _case(2, n=25, T=0.28)
    rng = np.random.default_rng(3)
    dz = rng.normal(0, 1, (1, WT.shape[1]))
    gW, gt = OL.li_readout_grad(t, src, n, WT, q, dz)
    f = lambda tt, W: float(np.sum(OL.li_readout(tt, src, n, W, q) * dz))
    W64 = WT.astype(np.float64)
    for c in range(WT.shape[0]):
        for k in range(WT.shape[1]):
            h = 1e-4
            Wp, Wm = W64.copy(), W64.copy()
            Wp[c, k] += h
            Wm[c, k] -= h
            fd = (f(t.astype(np.float64), Wp) - f(t.astype(np.float64), Wm)) / (2 * h)
            assert abs(fd - gW[c, k]) <= 1e-8 * max(1.0, abs(fd))
    for e in range(t.shape[1]):
        h = 1e-7
        tp, tm_ = t.astype(np.float64), t.astype(np.float64)
        tp[0, e] += h
        tm_[0, e] -= h
        fd = (f(tp, W64) - f(tm_, W64)) / (2 * h)
        assert abs(fd - gt[0, e]) <= 1e-5 * max(1e-3, abs(fd)), (e, fd, gt[0, e])


def test_ce_with_temperature_against_torch():
    rng = np.random.default_rng(5)
    z = rng.normal(0, 30, (6, 4))
    y = rng.integers(0, 4, 6)
    beta = 0.07
    loss, dz = OL.ce_with_temperature(z, y, beta)
    zt = torch.tensor(z, dtype=torch.float64, requires_grad=True)
    lt = torch.nn.functional.cross_entropy(beta * zt, torch.tensor(y))
    lt.backward()
    assert abs(loss - lt.item()) < 1e-13
    assert np.allclose(dz, zt.grad.numpy(), rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("seed", range(4))
def test_interval_vmax_against_dense_sampling(seed):
    rng = np.random.default_rng(seed)
    for _ in range(50):
        V0 = rng.uniform(-1.0, 1.2)
        I0 = rng.uniform(-3.0, 6.0)
        L = rng.uniform(1e-4, 0.05)
        vmax, u = OL.interval_vmax(TM, TS, V0, I0, L)
        s = np.linspace(0.0, L, 200001)
        V = V0 * np.exp(-s / TM) + KA * I0 * (np.exp(-s / TM) - np.exp(-s / TS))
        assert vmax >= V.max() - 1e-12
        assert vmax - V.max() < 1e-9
        assert 0.0 <= u <= L


def test_interval_table_against_superposition_with_resets():
    """The true start state of every interval and its maximum: the
    superposed input responses minus (theta - v_r) e^{-(t - t_s)/tau_m} per
    earlier spike s (hard reset as subtraction) and I as superposed
    currents; the maximum by dense sampling with the spikes of earlier
    intervals only."""
    P = oracle.LifParams(v_reset=-0.3)
    rng = np.random.default_rng(8)
    n = 30
    t = np.sort(rng.random(n) * 0.06).astype(np.float32)
    w = rng.uniform(0.3, 2.5, n).astype(np.float32)
    r = oracle.forward(t.reshape(1, -1), np.arange(n, dtype=np.int32).reshape(1, -1), np.array([n], np.int32),
                       w.reshape(-1, 1), P)
    ns = int(r.out_n[0, 0])
    assert ns >= 3
    st, sk = r.out_t[0, 0, :ns], r.out_k[0, 0, :ns]
    rows = OL.interval_table(t, n, w, st, sk, ns, TM, TS, P.v_th, P.v_reset, 0.1)
    assert len(rows) == n + 1 and sum(r_[6] for r_ in rows) == len(set(sk.tolist()))
    t64, w64 = t.astype(np.float64), w.astype(np.float64)
    for j, (a, b, V, I, vmax, u, spk) in enumerate(rows):
        before = np.arange(n) < j
        sp = sk < j
        Vs = _v_superposed(a + 1e-15, t64[before], w64[before]) if j > 0 else 0.0
        Vs -= (P.v_th - P.v_reset) * np.sum(np.exp(-(a - st[sp]) / TM))
        Is = float(np.sum(w64[before] * np.exp(-(a - t64[before]) / TS)))
        assert abs(V - Vs) < 1e-12 and abs(I - Is) < 1e-12, (j, V, Vs, I, Is)
        s = np.linspace(a, b, 20001)
        Vd = np.array([_v_superposed(x, t64[before], w64[before]) for x in s[::100]])
        Vd -= (P.v_th - P.v_reset) * np.exp(-(s[::100, None] - st[sp][None, :]) / TM).sum(axis=1)
        assert vmax >= Vd.max() - 1e-12 and vmax - Vd.max() < 1e-6
        if spk:
            assert vmax >= P.v_th - 1e-12


def test_spike_count_regulariser_by_hand():
    """Two samples, two neurons, hand-made interval tables (rows: t0, t1, V,
    I, V_max, u, spiked); target 2 spikes."""
    th = 1.0
    mk = lambda vmaxes, spk: [(0, 0, 0, 0, v, 0, s) for v, s in zip(vmaxes, spk)]
    tables = [[mk([0.5, 1.3, 0.9], [False, True, False]), mk([0.2, 0.4], [False, False])],
              [mk([1.2, 1.1, 0.7], [True, True, False]), mk([0.8, 1.4, 1.6], [False, True, True])]]
    counts = np.array([[1, 0], [2, 2]])
    rp = OL.RegParams(c_target=2.0, lam_reg=0.5, lam_over=0.25)
    L_reg, L_over, coef = OL.spike_count_reg(tables, counts, th, rp)
    # neuron 0: mean count 1.5 -> under gate 0.25, over gate 0
    #   under terms: sample 0 mean(0.5, 0.1) = 0.3; sample 1 mean(0.3) = 0.3
    # neuron 1: mean count 1 -> under gate 0.5, over gate 0
    #   under terms: sample 0 mean(0.8, 0.6) = 0.7; sample 1 mean(0.2) = 0.2
    L0 = 0.25 * 0.3
    L1 = 0.5 * (0.7 + 0.2) / 2
    assert abs(L_reg - (L0 + L1) / 2) < 1e-15
    # individual over-firing: counts above 2: none
    assert L_over == 0.0
    # dL/dV_max by finite differences of lam_reg L_reg + lam_over L_over
    def total(tb):
        a, b_, _ = OL.spike_count_reg(tb, counts, th, rp)
        return rp.lam_reg * a + rp.lam_over * b_
    for b in range(2):
        for i in range(2):
            for j in range(len(tables[b][i])):
                h = 1e-6
                tp = [[list(x) for x in row] for row in tables]
                tm_ = [[list(x) for x in row] for row in tables]
                rowp = list(tp[b][i][j]); rowp[4] += h; tp[b][i][j] = tuple(rowp)
                rowm = list(tm_[b][i][j]); rowm[4] -= h; tm_[b][i][j] = tuple(rowm)
                fd = (total(tp) - total(tm_)) / (2 * h)
                assert abs(fd - coef[b][i][j]) < 1e-8, (b, i, j, fd, coef[b][i][j])


def test_individual_over_firing_term_by_hand():
    th = 1.0
    mk = lambda vmaxes, spk: [(0, 0, 0, 0, v, 0, s) for v, s in zip(vmaxes, spk)]
    tables = [[mk([1.5, 1.2, 1.1, 0.2], [True, True, True, False])]]
    counts = np.array([[3]])
    rp = OL.RegParams(c_target=2.0)
    L_reg, L_over, _ = OL.spike_count_reg(tables, counts, th, rp)
    over = (0.5 + 0.2 + 0.1) / 3
    assert abs(L_over - 0.5 * over) < 1e-15            # gate 3/2 - 1, one neuron
    assert abs(L_reg - 0.5 * over) < 1e-15             # batch of one: same gate


def _reg_loss(ev, WT, P, rp):
    """lam_reg L_reg + lam_over L_over of the layer's own forward at WT."""
    r = oracle.forward(ev.ev_t, ev.ev_src, ev.ev_n, WT, P)
    L_reg, L_over, _, _, _ = OL.spike_count_reg_grad(ev.ev_t, ev.ev_src, ev.ev_n, WT, r.out_t, r.out_k, r.out_n,
                                                    P.tau_mem, P.tau_syn, P.v_th, P.v_reset, P.t_end, rp)
    return rp.lam_reg * L_reg + rp.lam_over * L_over, r.out_n


@pytest.mark.parametrize("vr", [0.0, -0.3])
def test_regulariser_gradients_match_finite_differences(vr):
    """App. E.1 regularisers: the direct V_max terms plus the layer's backward
    pass of the spike-time terms against central differences of the loss
    recomputed from a fresh forward (float64 weights and times; gates and
    interval sets unchanged by the small steps)."""
    cfg = W.random_small(51, B=3, C=12, N=6, n_events=60, T=0.15, gain=10.0)
    ev = cfg.events
    WT = cfg.layers[0].WT.astype(np.float64)
    P = oracle.LifParams(solver_reg=0.0, v_reset=vr)
    rp = OL.RegParams(c_target=3.0, lam_reg=0.7, lam_over=0.4)
    r = oracle.forward(ev.ev_t, ev.ev_src, ev.ev_n, WT.astype(np.float32), P)
    assert r.out_n.max() > 3 and (r.out_n.mean(axis=0) < 3).any() and (r.out_n.mean(axis=0) > 3).any()
    L_reg, L_over, gWd, gTd, gS = OL.spike_count_reg_grad(ev.ev_t, ev.ev_src, ev.ev_n, WT.astype(np.float32),
                                                         r.out_t, r.out_k, r.out_n, P.tau_mem, P.tau_syn, P.v_th,
                                                         P.v_reset, P.t_end, rp)
    gWs, gTs = oracle.backward(ev.ev_t, ev.ev_src, ev.ev_n, WT.astype(np.float32), r, gS, P)
    gW, gT = gWd + gWs, gTd + gTs
    assert np.abs(gW).max() > 0 and np.abs(gS).max() > 0
    # weights: the oracle reads float32 weights, so perturb in a way float32 holds exactly
    checked = 0
    for c in range(WT.shape[0]):
        for i in range(WT.shape[1]):
            h = 2.0 ** -14
            Wp, Wm = WT.copy(), WT.copy()
            Wp[c, i] += h
            Wm[c, i] -= h
            lp, np_ = _reg_loss(ev, Wp.astype(np.float32), P, rp)
            lm, nm = _reg_loss(ev, Wm.astype(np.float32), P, rp)
            if not (np.array_equal(np_, r.out_n) and np.array_equal(nm, r.out_n)):
                continue
            fd = (lp - lm) / (2 * h)
            assert abs(fd - gW[c, i]) <= 2e-4 * max(abs(fd), 1e-2 * np.abs(gW).max()), (c, i, fd, gW[c, i])
            checked += 1
    assert checked >= 50
    # input times (float32 steps of 2^-20 s)
    done = 0
    for b in range(ev.B):
        for k in range(0, int(ev.ev_n[b]), 7):
            h = 2.0 ** -20
            tp, tm_ = ev.ev_t.copy(), ev.ev_t.copy()
            tp[b, k] += h
            tm_[b, k] -= h
            if (k + 1 < ev.ev_n[b] and tp[b, k] >= ev.ev_t[b, k + 1]) or (k > 0 and tm_[b, k] <= ev.ev_t[b, k - 1]):
                continue
            lp, np_ = _reg_loss(W.EventBatch(tp, ev.ev_src, ev.ev_n), WT.astype(np.float32), P, rp)
            lm, nm = _reg_loss(W.EventBatch(tm_, ev.ev_src, ev.ev_n), WT.astype(np.float32), P, rp)
            if not (np.array_equal(np_, r.out_n) and np.array_equal(nm, r.out_n)):
                continue
            fd = (lp - lm) / (2 * h)
            assert abs(fd - gT[b, k]) <= 2e-3 * max(abs(fd), 1e-2 * np.abs(gT).max()), (b, k, fd, gT[b, k])
            done += 1
    assert done >= 10


def _dreg_loss(ev, WT, DT, P, rp):
    """lam_reg L_reg + lam_over L_over of a delayed layer's own forward."""
    r = oracle.forward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, WT, DT, P)
    q_t, q_k = oracle.delay_queues(ev.ev_t, ev.ev_src, ev.ev_n, DT)
    tables = OL.delayed_interval_tables(ev.ev_src, ev.ev_n, WT, q_t, q_k, r.out_t, r.out_k, r.out_n, P.tau_mem,
                                        P.tau_syn, P.v_th, P.v_reset, P.t_end)
    L_reg, L_over, _ = OL.spike_count_reg(tables, r.out_n, P.v_th, rp)
    return rp.lam_reg * L_reg + rp.lam_over * L_over, r.out_n, q_k


def test_delayed_regulariser_tables_reduce_to_the_plain_ones():
    """With zero delays every neuron's queue is the sample's own event order
    (arrivals t_k, ties by k), so the delayed tables are the plain ones."""
    cfg = W.random_small(53, B=2, C=10, N=5, n_events=50, T=0.15, gain=10.0)
    ev = cfg.events
    WT = cfg.layers[0].WT
    P = oracle.LifParams(v_reset=-0.3)
    r = oracle.forward(ev.ev_t, ev.ev_src, ev.ev_n, WT, P)
    q_t, q_k = oracle.delay_queues(ev.ev_t, ev.ev_src, ev.ev_n, np.zeros_like(WT))
    tab_d = OL.delayed_interval_tables(ev.ev_src, ev.ev_n, WT, q_t, q_k, r.out_t, r.out_k, r.out_n, P.tau_mem,
                                       P.tau_syn, P.v_th, P.v_reset, P.t_end)
    rp = OL.RegParams(c_target=3.0, lam_reg=0.7, lam_over=0.4)
    a = OL.spike_count_reg_grad(ev.ev_t, ev.ev_src, ev.ev_n, WT, r.out_t, r.out_k, r.out_n, P.tau_mem, P.tau_syn,
                                P.v_th, P.v_reset, P.t_end, rp)
    d = OL.spike_count_reg_delayed_grad(ev.ev_t, ev.ev_src, ev.ev_n, WT, q_t, q_k, r.out_t, r.out_k, r.out_n,
                                        P.tau_mem, P.tau_syn, P.v_th, P.v_reset, P.t_end, rp)
    for b in range(ev.B):
        for i in range(WT.shape[1]):
            n = int(ev.ev_n[b])
            plain = OL.interval_table(ev.ev_t[b, :n], n, WT[ev.ev_src[b, :n], i], r.out_t[b, i], r.out_k[b, i],
                                      int(r.out_n[b, i]), P.tau_mem, P.tau_syn, P.v_th, P.v_reset, P.t_end)
            assert tab_d[b][i] == plain
    assert d[0] == a[0] and d[1] == a[1]
    assert np.allclose(d[2], a[2], rtol=1e-12, atol=0) and np.allclose(d[4], a[3], rtol=1e-12, atol=1e-300)
    assert np.array_equal(d[5], a[4])
    # with zero delays dL/dd_{j,i} sums the arrival terms of channel j's events at neuron i
    assert np.abs(d[3]).max() > 0


@pytest.mark.parametrize("vr", [0.0, -0.3])
def test_delayed_regulariser_gradients_match_finite_differences(vr):
    """The regularisers of a layer with synaptic delays: the direct terms plus
    the delayed layer's backward pass of the spike-time terms against central
    differences of the loss from a fresh delayed forward, for weights, delays
    and input times (steps float32 holds exactly; cases whose spike counts or
    queue order the step changes are skipped)."""
    cfg = W.random_small(52, B=3, C=12, N=6, n_events=60, T=0.15, gain=10.0)
    ev = cfg.events
    WT = cfg.layers[0].WT.astype(np.float32)
    DT = W.uniform_delays(52, 12, 6, d_max=0.03)
    P = oracle.LifParams(solver_reg=0.0, v_reset=vr)
    rp = OL.RegParams(c_target=3.0, lam_reg=0.7, lam_over=0.4)
    r = oracle.forward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, WT, DT, P)
    assert r.out_n.max() > 3 and (r.out_n.mean(axis=0) < 3).any() and (r.out_n.mean(axis=0) > 3).any()
    q_t, q_k = oracle.delay_queues(ev.ev_t, ev.ev_src, ev.ev_n, DT)
    L_reg, L_over, gWd, gDd, gTd, gS = OL.spike_count_reg_delayed_grad(
        ev.ev_t, ev.ev_src, ev.ev_n, WT, q_t, q_k, r.out_t, r.out_k, r.out_n, P.tau_mem, P.tau_syn, P.v_th,
        P.v_reset, P.t_end, rp)
    gWs, gDs, gTs = oracle.backward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, WT, DT, r, gS, P)
    gW, gD, gT = gWd + gWs, gDd + gDs, gTd + gTs
    assert np.abs(gW).max() > 0 and np.abs(gD).max() > 0 and np.abs(gS).max() > 0

    def same(res):
        return np.array_equal(res[1], r.out_n) and np.array_equal(res[2], q_k)

    checked = {"W": 0, "D": 0, "t": 0}
    for c in range(WT.shape[0]):
        for i in range(WT.shape[1]):
            for name, base, h, g in (("W", WT, 2.0 ** -14, gW), ("D", DT, 2.0 ** -20, gD)):
                xp, xm = base.copy(), base.copy()
                xp[c, i] += np.float32(h)
                xm[c, i] -= np.float32(h)
                if name == "D" and xm[c, i] < 0:
                    continue
                rp_ = _dreg_loss(ev, xp, DT, P, rp) if name == "W" else _dreg_loss(ev, WT, xp, P, rp)
                rm_ = _dreg_loss(ev, xm, DT, P, rp) if name == "W" else _dreg_loss(ev, WT, xm, P, rp)
                if not (same(rp_) and same(rm_)):
                    continue
                fd = (rp_[0] - rm_[0]) / (2 * h)
                tol = 2e-4 if name == "W" else 2e-3
                assert abs(fd - g[c, i]) <= tol * max(abs(fd), 1e-2 * np.abs(g).max()), (name, c, i, fd, g[c, i])
                checked[name] += 1
    for b in range(ev.B):
        for k in range(0, int(ev.ev_n[b]), 5):
            h = 2.0 ** -20
            tp, tm_ = ev.ev_t.copy(), ev.ev_t.copy()
            tp[b, k] += h
            tm_[b, k] -= h
            if (k + 1 < ev.ev_n[b] and tp[b, k] >= ev.ev_t[b, k + 1]) or (k > 0 and tm_[b, k] <= ev.ev_t[b, k - 1]):
                continue
            rp_ = _dreg_loss(W.EventBatch(tp, ev.ev_src, ev.ev_n), WT, DT, P, rp)
            rm_ = _dreg_loss(W.EventBatch(tm_, ev.ev_src, ev.ev_n), WT, DT, P, rp)
            if not (same(rp_) and same(rm_)):
                continue
            fd = (rp_[0] - rm_[0]) / (2 * h)
            assert abs(fd - gT[b, k]) <= 2e-3 * max(abs(fd), 1e-2 * np.abs(gT).max()), (b, k, fd, gT[b, k])
            checked["t"] += 1
    assert checked["W"] >= 40 and checked["D"] >= 30 and checked["t"] >= 10, checked
