"""GPU parity of the paper's readout and loss (lif_li_readout) and of the
gradient scatter through the merge (lif_merge_grad), through the C ABI,
against the float64 oracle (oracle/loss.py) on identical float32 inputs."""
import math

import numpy as np
import pytest

import oracle
import workloads as W
from oracle import loss as OL

pytestmark = pytest.mark.gpu

LOGIT_RTOL = 1e-6          # float32 outputs of float64 sums
GRAD_RTOL = 1e-4           # the gradient tolerance of the parity bar


@pytest.fixture(scope="module")
def env():
    import torch
    import paper_2603_13283_amd as lif
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    lif.load()
    return torch, lif


def _dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda:0")


def _close(got, ref, rtol, label):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = max(np.abs(ref).max(), 1e-30)
    err = np.abs(got - ref) - rtol * np.abs(ref)
    bad = np.argwhere(err > rtol * 1e-2 * scale)
    assert len(bad) == 0, f"{label}: {len(bad)} elements off, first {tuple(bad[0])} gpu {got[tuple(bad[0])]} " \
                          f"oracle {ref[tuple(bad[0])]}"


def _queue(seed, B, C, n_events, T, empty_sample=True):
    ev = W.random_small(seed, B=B, C=C, N=2, n_events=n_events, T=T, gain=1.0).events
    if empty_sample:
        ev.ev_n[min(1, B - 1)] = 0
    return ev


def run_case(env, ev, WT, q: OL.LiParams, labels, label):
    torch, lif = env
    print(f"[case] {label} B={ev.B} E_max={ev.E_max} C={WT.shape[0]} classes={WT.shape[1]}", flush=True)
    lq = lif.LiParams(q.tau_mem, q.tau_syn, q.tau_li, q.tau_max, q.beta)
    args = [_dev(torch, a) for a in (ev.ev_t, ev.ev_src, ev.ev_n, WT)]
    z, loss, gW, gT = lif.li_readout(*args, lq, labels=_dev(torch, labels))
    torch.cuda.synchronize()
    zr = OL.li_readout(ev.ev_t, ev.ev_src, ev.ev_n, WT, q)
    lr, dz = OL.ce_with_temperature(zr, labels, q.beta)
    gWr, gTr = OL.li_readout_grad(ev.ev_t, ev.ev_src, ev.ev_n, WT, q, dz)
    _close(z.cpu().numpy(), zr, LOGIT_RTOL, f"{label} logits")
    assert abs(loss.item() - lr) <= LOGIT_RTOL * max(1.0, abs(lr)), (loss.item(), lr)
    _close(gW.cpu().numpy(), gWr, GRAD_RTOL, f"{label} grad_WT")
    _close(gT.cpu().numpy(), gTr, GRAD_RTOL, f"{label} grad_ev_t")
    # bitwise reproducible: a second call gives the same bits
    z2, loss2, gW2, gT2 = lif.li_readout(*args, lq, labels=_dev(torch, labels))
    for a, b_ in ((z, z2), (loss, loss2), (gW, gW2), (gT, gT2)):
        assert torch.equal(a.view(torch.int32), b_.view(torch.int32))
    return z, zr


@pytest.mark.parametrize("tau_li", [0.5, math.inf])
def test_readout_small_ragged(env, tau_li):
    ev = _queue(3, B=6, C=300, n_events=1500, T=1.0)
    rng = np.random.default_rng(4)
    WT = (rng.normal(0, 1, (300, 20)) * 4 / math.sqrt(300)).astype(np.float32)
    labels = rng.integers(0, 20, 6).astype(np.int32)
    q = OL.LiParams(tau_li=tau_li, tau_max=0.8, beta=0.5)
    assert (ev.ev_t[ev.ev_n > 0][:, 0] < 0.8).all() and (ev.ev_t.max() > 0.8)     # events past the window too
    z, _ = run_case(env, ev, WT, q, labels, f"ragged tau_li={tau_li}")
    assert (z[1] == 0).all()                                                       # the empty sample


@pytest.mark.parametrize("ncls", [1, 64])
def test_readout_class_counts(env, ncls):
    ev = _queue(5, B=3, C=50, n_events=400, T=0.5, empty_sample=False)
    rng = np.random.default_rng(ncls)
    WT = rng.normal(0, 0.5, (50, ncls)).astype(np.float32)
    labels = rng.integers(0, ncls, 3).astype(np.int32)
    run_case(env, ev, WT, OL.LiParams(tau_li=0.2, tau_max=0.6, beta=0.2), labels, f"classes={ncls}")


def test_readout_on_a_merged_hidden_layer(env):
    """The readout of config 3's shape: the spikes of a 700 -> 512 layer
    merged into a queue, 512 -> 20 classes; the oracle on sampled rows."""
    torch, lif = env
    cfg = W.config3()
    B = 16
    ev = cfg.events
    args = [_dev(torch, a[:B]) for a in (ev.ev_t, ev.ev_src, ev.ev_n)]
    P = lif.Params(s_max=128)
    out = lif.forward(*args, _dev(torch, cfg.layers[0].WT), P)
    E2 = 16384
    t2, s2, n2, perm, st = lif.merge(out, E2)
    torch.cuda.synchronize()
    rng = np.random.default_rng(7)
    WT = (rng.normal(0, 1, (512, 20)) * 4 / math.sqrt(512)).astype(np.float32)
    labels = rng.integers(0, 20, B).astype(np.int32)
    q = OL.LiParams(tau_li=0.5, tau_max=1.0, beta=0.05)
    lq = lif.LiParams(q.tau_mem, q.tau_syn, q.tau_li, q.tau_max, q.beta)
    z, loss, gW, gT = lif.li_readout(t2, s2, n2, _dev(torch, WT), lq, labels=_dev(torch, labels))
    torch.cuda.synchronize()
    t2n, s2n, n2n = t2.cpu().numpy(), s2.cpu().numpy(), n2.cpu().numpy()
    print(f"[case] merged queue lengths {n2n.min()}..{n2n.max()}", flush=True)
    assert n2n.min() > 100
    zr = OL.li_readout(t2n, s2n, n2n, WT, q)
    lr, dz = OL.ce_with_temperature(zr, labels, q.beta)
    _close(z.cpu().numpy(), zr, LOGIT_RTOL, "merged logits")
    assert abs(loss.item() - lr) <= LOGIT_RTOL * max(1.0, abs(lr))
    rows = [0, 5, 11]
    gWr, gTr = OL.li_readout_grad(t2n, s2n, n2n, WT, q, dz)
    _close(gW.cpu().numpy(), gWr, GRAD_RTOL, "merged grad_WT")
    _close(gT.cpu().numpy()[rows], gTr[rows], GRAD_RTOL, "merged grad_ev_t")
    # the queue-time gradient routed back to the layer's spikes
    g_out = lif.merge_grad(gT, perm, n2, 512, 128)
    torch.cuda.synchronize()
    go, pn, gTn = g_out.cpu().numpy(), perm.cpu().numpy(), gT.cpu().numpy()
    ref = np.zeros((B, 512 * 128), np.float32)
    for b in range(B):
        k = n2n[b]
        ref[b, pn[b, :k]] = gTn[b, :k]
    assert np.array_equal(go.reshape(B, -1), ref)


def _reg_oracle(ev, WT, r, P, c_target):
    """The oracle's interval tables from its own spike trains, and the
    regulariser terms."""
    B, N = r.out_n.shape
    tables = []
    for b in range(B):
        n = int(ev.ev_n[b])
        row = []
        for i in range(N):
            ns = int(r.out_n[b, i])
            w = WT[ev.ev_src[b, :n], i]
            row.append(OL.interval_table(ev.ev_t[b, :n], n, w, r.out_t[b, i, :ns], r.out_k[b, i, :ns], ns, P.tau_mem,
                                         P.tau_syn, P.v_th, P.v_reset, P.t_end))
        tables.append(row)
    L_reg, L_over, _ = OL.spike_count_reg(tables, r.out_n, P.v_th, OL.RegParams(c_target=c_target))
    under = np.array([[np.mean([max(P.v_th - x[4], 0.0) for x in t if not x[6]] or [0.0]) for t in row]
                      for row in tables])
    over = np.array([[np.mean([max(x[4] - P.v_th, 0.0) for x in t if x[6]] or [0.0]) for t in row]
                     for row in tables])
    return L_reg, L_over, under, over


@pytest.mark.parametrize("t_end,vr", [(math.inf, 0.0), (0.5, -0.3)])
def test_spike_count_regularisers(env, t_end, vr):
    """App. E.1 on a driven layer with ragged queues and an empty sample: the
    per-(sample, neuron) hinge means and both loss terms, from the oracle's
    spike trains handed to both sides (rounded to float32 for the GPU)."""
    torch, lif = env
    cfg = W.random_small(51, B=4, C=40, N=70, n_events=600, T=0.4, gain=6.0)
    ev, WT = cfg.events, cfg.layers[0].WT
    ev.ev_n[2] = 0
    P = oracle.LifParams(s_max=64, t_end=t_end, v_reset=vr)
    r = oracle.forward(ev.ev_t, ev.ev_src, ev.ev_n, WT, P)
    assert r.out_n.sum() > 100 and not r.capped.any()
    print(f"[case] regularisers t_end={t_end} v_reset={vr} spikes={int(r.out_n.sum())}", flush=True)
    L_reg, L_over, under, over = _reg_oracle(ev, WT, r, P, 4.0)
    fwd = lif.ForwardOut(_dev(torch, r.out_t.astype(np.float32)), _dev(torch, r.out_n),
                         _dev(torch, r.out_i.astype(np.float32)), None, _dev(torch, r.out_k))
    args = [_dev(torch, a) for a in (ev.ev_t, ev.ev_src, ev.ev_n, WT)]
    lp = lif.Params(s_max=64, t_end=t_end, v_reset=vr)
    loss, gu, go = lif.spike_count_reg(*args, fwd, 4.0, lp)
    loss2, _, _ = lif.spike_count_reg(*args, fwd, 4.0, lp)
    torch.cuda.synchronize()
    _close(gu.cpu().numpy(), under, 1e-5, "under")
    _close(go.cpu().numpy(), over, 1e-5, "over")
    assert (gu.cpu().numpy()[2] == P.v_th).all()            # the empty sample: V = 0 throughout
    assert abs(loss[0].item() - L_reg) <= 1e-5 * abs(L_reg), (loss[0].item(), L_reg)
    assert abs(loss[1].item() - L_over) <= 1e-5 * max(abs(L_over), 1e-12), (loss[1].item(), L_over)
    assert torch.equal(loss.view(torch.int32), loss2.view(torch.int32))


@pytest.mark.parametrize("t_end,vr", [(math.inf, 0.0), (0.5, -0.3)])
def test_spike_count_regulariser_gradients(env, t_end, vr):
    """The gradient of lam_reg L_reg + lam_over L_over: the loss values, the
    upstream spike-time gradient and the direct weight and input-time parts
    against the oracle on identical inputs (the oracle's spike trains in
    float32), then the full weight and input-time gradients through the
    layer's backward pass."""
    from tests.parity import compare_grad
    torch, lif = env
    cfg = W.random_small(51, B=4, C=40, N=70, n_events=600, T=0.4, gain=6.0)
    ev, WT = cfg.events, cfg.layers[0].WT
    ev.ev_n[2] = 0
    P = oracle.LifParams(s_max=64, t_end=t_end, v_reset=vr)
    r = oracle.forward(ev.ev_t, ev.ev_src, ev.ev_n, WT, P)
    assert r.out_n.sum() > 100 and not r.capped.any()
    c_target = float(np.median(r.out_n.mean(axis=0))) + 0.5
    rp = OL.RegParams(c_target=c_target, lam_reg=0.8, lam_over=0.3)
    r32 = r.rounded()
    print(f"[case] regulariser gradients t_end={t_end} v_reset={vr} spikes={int(r.out_n.sum())} "
          f"c_target={c_target}", flush=True)
    L_reg, L_over, gWd, gTd, gS = OL.spike_count_reg_grad(ev.ev_t, ev.ev_src, ev.ev_n, WT, r32.out_t, r.out_k,
                                                         r.out_n, P.tau_mem, P.tau_syn, P.v_th, P.v_reset, P.t_end, rp)
    gWs, gTs = oracle.backward(ev.ev_t, ev.ev_src, ev.ev_n, WT, r32, gS, P)
    fwd = lif.ForwardOut(_dev(torch, r32.out_t.astype(np.float32)), _dev(torch, r.out_n),
                         _dev(torch, r32.out_i.astype(np.float32)), None, _dev(torch, r.out_k))
    args = [_dev(torch, a) for a in (ev.ev_t, ev.ev_src, ev.ev_n, WT)]
    lp = lif.Params(s_max=64, t_end=t_end, v_reset=vr)
    seed = torch.full((ev.B, WT.shape[1], 64), 0.25, device="cuda:0") * fwd.out_t.isfinite()
    loss, gsp, gW, gT = lif.spike_count_reg_backward(*args, fwd, c_target, 0.8, 0.3, lp, grad_spike=seed.clone())
    torch.cuda.synchronize()
    assert abs(loss[0].item() - L_reg) <= 1e-5 * abs(L_reg) and abs(loss[1].item() - L_over) <= 1e-5 * max(
        abs(L_over), 1e-12)
    g_spike = (gsp - seed).cpu().numpy()
    assert np.abs(gS).max() > 0 and np.abs(gWd).max() > 0
    es = compare_grad(g_spike, gS, label="regulariser spike-time gradient")
    ew = compare_grad(gW.cpu().numpy(), gWd, label="regulariser direct grad_W")
    et = compare_grad(gT.cpu().numpy(), gTd, label="regulariser direct grad_t")
    # the full gradient: direct part plus the layer's backward of the spike-time part
    bW, bT = lif.backward(*args, fwd, gsp - seed, lp)
    torch.cuda.synchronize()
    fw = compare_grad((gW + bW).cpu().numpy(), gWd + gWs, label="regulariser grad_W")
    ft = compare_grad((gT + bT).cpu().numpy(), gTd + gTs, label="regulariser grad_t")
    print(f"    rel spike {es:.2e} direct W {ew:.2e} t {et:.2e}; full W {fw:.2e} t {ft:.2e}", flush=True)
    # bitwise reproducible
    loss2, gsp2, gW2, gT2 = lif.spike_count_reg_backward(*args, fwd, c_target, 0.8, 0.3, lp, grad_spike=seed.clone())
    for a, b_ in ((loss, loss2), (gsp, gsp2), (gW, gW2), (gT, gT2)):
        assert torch.equal(a.view(torch.int32), b_.view(torch.int32))
