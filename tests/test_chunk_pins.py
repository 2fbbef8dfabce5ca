"""Pins of the chunk-mode oracle (Sec. 3.2.1 speculative execution with a
fixed budget of C chunk iterations): with a budget that suffices it gives the
serial event loop's spikes bit for bit; its work counters (Appendix G) and,
under a budget that runs out, its truncated spike trains and consumed counts
agree with a bookkeeping of chunk positions written from the definition over
the serial loop's spike list."""
import numpy as np
import pytest

import oracle
import workloads as W


def bookkeeping(n, ks, K, C, s_max):
    """Chunk iterations over a queue of n events for a neuron whose serial
    spike train has consumed-event counts ks: each iteration covers events
    p .. min(p + K, n) - 1; it ends at the first spike whose interval it
    reaches (an interval closed by one of its events, or the one after the
    last event when it holds it), the next iteration starting at that
    spike's pending event; without one, its events are consumed.  Returns
    (spikes found, consumed, processed)."""
    p, si, processed, chunks = 0, 0, 0, 0
    while chunks < C:
        chunks += 1
        end = min(p + K, n)
        processed += end - p
        if si < len(ks) and (ks[si] < end or (end == n and ks[si] <= n)):
            p = int(ks[si])
            si += 1
            if si >= s_max:
                break
            continue
        if end == n:
            p = n
            break
        p = end
    return si, p, processed


@pytest.mark.parametrize("K", [1, 4, 64, 128])
def test_chunked_matches_serial_with_enough_budget(K):
    cfg = W.random_small(61, B=3, C=30, N=40, n_events=500, T=0.4, gain=12.0)
    ev, WT = cfg.events, cfg.layers[0].WT
    P = oracle.LifParams(s_max=64)
    r = oracle.forward(ev.ev_t, ev.ev_src, ev.ev_n, WT, P)
    C = 10 ** 6
    q, consumed, processed = oracle.forward_chunked(ev.ev_t, ev.ev_src, ev.ev_n, WT, K, C, P)
    assert np.array_equal(q.out_n, r.out_n) and np.array_equal(q.out_k, r.out_k)
    assert np.array_equal(q.out_t, r.out_t) and np.array_equal(q.out_i, r.out_i)
    assert r.out_n.sum() > 100
    for b in range(ev.B):
        for i in range(WT.shape[1]):
            ns = int(r.out_n[b, i])
            found, cons, proc = bookkeeping(int(ev.ev_n[b]), r.out_k[b, i, :ns], K, C, P.s_max)
            assert found == ns
            if not r.capped[b, i]:
                assert cons == ev.ev_n[b] == consumed[b, i]
            assert proc == processed[b, i], (b, i, proc, processed[b, i])
    # a larger chunk never processes fewer events than it consumes
    assert (processed >= consumed).all()


@pytest.mark.parametrize("K,C", [(16, 5), (64, 3), (8, 40)])
def test_chunked_budget_truncates(K, C):
    """A budget that runs out: the spikes are the first ones of the serial
    train, and the consumed and processed counts follow the bookkeeping."""
    cfg = W.random_small(62, B=2, C=30, N=40, n_events=400, T=0.4, gain=14.0)
    ev, WT = cfg.events, cfg.layers[0].WT
    P = oracle.LifParams(s_max=64)
    r = oracle.forward(ev.ev_t, ev.ev_src, ev.ev_n, WT, P)
    q, consumed, processed = oracle.forward_chunked(ev.ev_t, ev.ev_src, ev.ev_n, WT, K, C, P)
    truncated = 0
    for b in range(ev.B):
        for i in range(WT.shape[1]):
            ns = int(r.out_n[b, i])
            found, cons, proc = bookkeeping(int(ev.ev_n[b]), r.out_k[b, i, :ns], K, C, P.s_max)
            assert q.out_n[b, i] == found
            assert np.array_equal(q.out_t[b, i, :found], r.out_t[b, i, :found])
            assert consumed[b, i] == cons and processed[b, i] == proc
            truncated += cons < ev.ev_n[b]
    assert truncated > 0, "the budget must run out for some neurons"


def test_chunked_silent_neuron_counts():
    """A silent neuron consumes its whole queue in ceil(n / K) iterations."""
    ev = W.random_small(63, B=1, C=10, N=3, n_events=300, T=0.3, gain=0.0).events
    WT = np.zeros((10, 3), np.float32)
    q, consumed, processed = oracle.forward_chunked(ev.ev_t, ev.ev_src, ev.ev_n, WT, 64, 10 ** 6,
                                                    oracle.LifParams())
    n = int(ev.ev_n[0])
    assert (q.out_n == 0).all() and (consumed == n).all() and (processed == n).all()
    q, consumed, processed = oracle.forward_chunked(ev.ev_t, ev.ev_src, ev.ev_n, WT, 64, 2, oracle.LifParams())
    assert (consumed == min(n, 128)).all() and (processed == min(n, 128)).all()
