"""Pins of the delayed-layer oracle (Sec. 3.1 Eq. spike_input: each input
spike reaches neuron i after its synapse's delay d_ij; App. E.2: a sorted
event queue per neuron).  Each pin checks the oracle against something other
than itself: the plain layer it must reduce to, numpy's sort, the time
translation invariance of the dynamics, and central finite differences of
the pure-Python reference."""
import math

import numpy as np
import pytest

import oracle
import workloads as W
from oracle import ref


def _case(seed, B=3, C=40, N=12, n=300, T=0.4, gain=10.0, d_max=0.1):
    cfg = W.random_small(seed, B=B, C=C, N=N, n_events=n, T=T, gain=gain)
    return cfg.events, cfg.layers[0].WT, W.uniform_delays(seed, C, N, d_max)


def test_zero_delays_reduce_to_the_layer():
    """With every d_ij = 0 the queues are the sample's queue and the layer is
    the plain one: identical spikes and identical weight and time gradients;
    the delay gradient of neuron i summed over channels then equals the time
    gradient summed over the events (both are sums of the same dL/da)."""
    ev, WT, _ = _case(1)
    DT = np.zeros_like(WT)
    P = oracle.LifParams(solver_reg=0.0)
    r0 = oracle.forward(ev.ev_t, ev.ev_src, ev.ev_n, WT, P)
    r1 = oracle.forward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, WT, DT, P)
    assert r0.out_n.sum() > 30
    for a, b in ((r0.out_t, r1.out_t), (r0.out_i, r1.out_i), (r0.out_n, r1.out_n), (r0.out_k, r1.out_k)):
        assert np.array_equal(a, b)
    g = np.random.default_rng(2).standard_normal(r0.out_t.shape) * np.isfinite(r0.out_t)
    gW0, gT0 = oracle.backward(ev.ev_t, ev.ev_src, ev.ev_n, WT, r0, g, P, nthreads=1)
    gW1, gD1, gT1 = oracle.backward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, WT, DT, r1, g, P, nthreads=1)
    assert np.array_equal(gW0, gW1) and np.array_equal(gT0, gT1)
    tot_t = sum(gT1[b, : ev.ev_n[b]].sum() for b in range(ev.B))
    assert abs(gD1.sum() - tot_t) <= 1e-12 * max(1.0, np.abs(gD1).sum())


def test_queues_against_numpy_sort():
    """Each neuron's queue is the sample's events ordered by the float32
    arrival t_k + d_ij, equal arrivals in event order."""
    ev, _, DT = _case(3, B=4, C=25, N=9, n=200)
    q_t, q_k = oracle.delay_queues(ev.ev_t, ev.ev_src, ev.ev_n, DT)
    for b in range(ev.B):
        n = int(ev.ev_n[b])
        t, s = ev.ev_t[b, :n], ev.ev_src[b, :n]
        for i in range(DT.shape[1]):
            a = t + DT[s, i]                           # float32 + float32 in numpy: float32
            assert a.dtype == np.float32
            order = np.lexsort((np.arange(n), a))
            assert np.array_equal(q_k[b, i, :n], order)
            assert np.array_equal(q_t[b, i, :n], a[order])


def test_ties_keep_event_order():
    """Equal arrivals from different channels keep the sample's order."""
    t = np.array([0.25, 0.5, 0.5, 0.75], np.float32)
    src = np.array([0, 1, 2, 0], np.int32)
    ev = W.pack_events([t], [src])
    DT = np.array([[0.25], [0.0], [0.0]], np.float32)     # event 0 arrives at 0.5 with events 1, 2
    q_t, q_k = oracle.delay_queues(ev.ev_t, ev.ev_src, ev.ev_n, DT)
    assert list(q_k[0, 0]) == [0, 1, 2, 3]
    assert list(q_t[0, 0]) == [0.5, 0.5, 0.5, 1.0]


def test_each_neuron_is_the_plain_layer_on_its_own_queue():
    """Neuron i of the delayed layer equals a one-neuron plain layer fed the
    queue built here with numpy (times t_k + d_ij, sorted)."""
    ev, WT, DT = _case(5, B=2, C=30, N=6, n=250, gain=12.0)
    P = oracle.LifParams(v_reset=-0.2)
    r = oracle.forward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, WT, DT, P)
    assert r.out_n.sum() > 20
    for b in range(ev.B):
        n = int(ev.ev_n[b])
        t, s = ev.ev_t[b, :n], ev.ev_src[b, :n]
        for i in range(WT.shape[1]):
            a = t + DT[s, i]
            o = np.lexsort((np.arange(n), a))
            one = W.EventBatch(a[o][None, :], s[o][None, :].astype(np.int32), np.array([n], np.int32))
            r1 = oracle.forward(one.ev_t, one.ev_src, one.ev_n, WT[:, i:i + 1], P)
            assert np.array_equal(r1.out_t[0, 0], r.out_t[b, i])
            assert np.array_equal(r1.out_k[0, 0], r.out_k[b, i])


def test_uniform_delay_shifts_every_spike():
    """All synapses with the same delay c: the neuron rests until the first
    arrival, so its spike train is the undelayed one shifted by c (times and
    c on a 2^-20 grid, so every float32 sum is exact)."""
    rng = np.random.default_rng(7)
    C, N, n = 20, 8, 200
    t = (rng.integers(0, 2 ** 18, n) * 2.0 ** -20).astype(np.float32)
    src = rng.integers(0, C, n).astype(np.int32)
    ev = W.pack_events([t], [src])
    WT = (rng.standard_normal((C, N)) * 12 / math.sqrt(C)).astype(np.float32)
    c = 0.03125
    DT = np.full((C, N), c, np.float32)
    r0 = oracle.forward(ev.ev_t, ev.ev_src, ev.ev_n, WT)
    r1 = oracle.forward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, WT, DT)
    assert r0.out_n.sum() > 10
    assert np.array_equal(r0.out_n, r1.out_n) and np.array_equal(r0.out_k, r1.out_k)
    m = np.isfinite(r0.out_t)
    assert np.allclose(r1.out_t[m], r0.out_t[m] + c, rtol=1e-12, atol=0)
    assert np.allclose(r1.out_i[m], r0.out_i[m], rtol=1e-12, atol=0)


def test_delay_gradient_sums_to_the_spike_gradient():
    """Shifting all of neuron i's arrivals by e shifts all its spikes by e
    (t_end = inf, no regularisation floor), so sum_j dL/dd_ij = sum_s g_is;
    shifting every input event shifts every spike: sum_k dL/dt_k = sum g."""
    ev, WT, DT = _case(11, B=2, C=30, N=10, n=260, gain=12.0)
    P = oracle.LifParams(solver_reg=0.0)
    r = oracle.forward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, WT, DT, P)
    assert r.out_n.sum() > 20
    g = np.random.default_rng(12).standard_normal(r.out_t.shape) * np.isfinite(r.out_t)
    gW, gD, gT = oracle.backward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, WT, DT, r, g, P)
    # per neuron (one sample at a time: gD sums over samples)
    for b in range(ev.B):
        one = W.EventBatch(ev.ev_t[b:b + 1], ev.ev_src[b:b + 1], ev.ev_n[b:b + 1])
        rb = r.select(np.arange(ev.B) == b)
        _, gDb, gTb = oracle.backward_delayed(one.ev_t, one.ev_src, one.ev_n, WT, DT, rb, g[b:b + 1], P)
        want = g[b].sum(axis=1)
        assert np.allclose(gDb.sum(axis=0), want, rtol=1e-9, atol=1e-9 * np.abs(g[b]).sum())
        assert abs(gTb.sum() - g[b].sum()) <= 1e-9 * max(1.0, np.abs(g[b]).sum())
    assert np.allclose(gD.sum(axis=0), g.sum(axis=(0, 2)), rtol=1e-9, atol=1e-9 * np.abs(g).sum())


def _ref_neuron_loss(times, src, d_col, w_col, g, n_max):
    a = np.asarray(times, np.float64) + np.asarray(d_col, np.float64)[src]
    o = np.lexsort((np.arange(len(a)), a))
    sp = ref.simulate(a[o], [w_col[c] for c in src[o]])
    return sum(g[s] * t for s, (t, _) in enumerate(sp[:n_max])), len(sp)


def test_delay_gradients_match_finite_differences():
    """dL/dd_ij, dL/dw_ij and dL/dt_k of L = sum_s g_s t_s against central
    differences of the pure-Python reference (bisection root, float64), on
    times and delays of a 2^-20 grid so that the float32 arrivals are exact."""
    rng = np.random.default_rng(21)
    C, N, n = 6, 3, 45
    t = (rng.integers(0, int(0.15 * 2 ** 20), n) * 2.0 ** -20).astype(np.float32)
    src = rng.integers(0, C, n).astype(np.int32)
    ev = W.pack_events([t], [src])
    t, src = ev.ev_t[0], ev.ev_src[0]
    WT = rng.uniform(-1.0, 4.0, (C, N)).astype(np.float32)
    DT = (rng.integers(0, int(0.03 * 2 ** 20), (C, N)) * 2.0 ** -20).astype(np.float32)
    P = oracle.LifParams(solver_reg=0.0)
    r = oracle.forward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, WT, DT, P)
    assert r.out_n.sum() >= 3
    g = rng.standard_normal(r.out_t.shape) * np.isfinite(r.out_t)
    gW, gD, gT = oracle.backward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, WT, DT, r, g, P)
    W64, D64, T64 = WT.astype(np.float64), DT.astype(np.float64), t.astype(np.float64)
    checked = 0
    for i in range(N):
        base = int(r.out_n[0, i])
        if base == 0:
            continue
        for c in range(C):
            if not (src == c).any():
                continue
            h = 1e-9
            Dp, Dm = D64[:, i].copy(), D64[:, i].copy()
            Dp[c] += h
            Dm[c] -= h
            lp, n_p = _ref_neuron_loss(T64, src, Dp, W64[:, i], g[0, i], base)
            lm, n_m = _ref_neuron_loss(T64, src, Dm, W64[:, i], g[0, i], base)
            assert n_p == n_m == base
            fd = (lp - lm) / (2 * h)
            assert abs(fd - gD[c, i]) <= 1e-5 * max(1.0, abs(fd)), (c, i, fd, gD[c, i])
            hw = 1e-6
            Wp, Wm = W64[:, i].copy(), W64[:, i].copy()
            Wp[c] += hw
            Wm[c] -= hw
            lp = _ref_neuron_loss(T64, src, D64[:, i], Wp, g[0, i], base)[0]
            lm = _ref_neuron_loss(T64, src, D64[:, i], Wm, g[0, i], base)[0]
            fdw = (lp - lm) / (2 * hw)
            assert abs(fdw - gW[c, i]) <= 1e-6 * max(1.0, abs(fdw)), (c, i, fdw, gW[c, i])
            checked += 1
    assert checked >= 6
    for k in range(0, n, 5):
        h = 1e-9
        tot = 0.0
        for sign in (1.0, -1.0):
            Tk = T64.copy()
            Tk[k] += sign * h
            tot += sign * sum(_ref_neuron_loss(Tk, src, D64[:, i], W64[:, i], g[0, i], int(r.out_n[0, i]))[0]
                              for i in range(N))
        fd = tot / (2 * h)
        assert abs(fd - gT[0, k]) <= 1e-5 * max(1.0, abs(fd)), (k, fd, gT[0, k])
