"""GPU parity of the layer with learnable synaptic delays (lif_delay_queues,
lif_layer_forward_delayed, lif_layer_backward_delayed) against the delayed
oracle on the same seeded inputs: the per-neuron queues bit for bit, the
spike trains, and the weight, delay and input-time gradients."""
import math

import numpy as np
import pytest

import oracle
import workloads as W
from tests.parity import compare_grad, compare_spikes

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch
    import paper_2603_13283_amd as lif
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    lif.load()
    return torch, lif


def _dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda:0")


def run_case(env, ev, WT, DT, label, P=None, OP=None, grads=True, twice=True):
    torch, lif = env
    P = P or lif.Params()
    OP = OP or oracle.LifParams()
    print(f"[case] {label} B={ev.B} E_max={ev.E_max} C={WT.shape[0]} N={WT.shape[1]}", flush=True)
    t, s, n, w, d = (_dev(torch, a) for a in (ev.ev_t, ev.ev_src, ev.ev_n, WT, DT))
    q = lif.delay_queues(t, s, n, d)
    out = lif.forward_delayed(q, s, n, w, P)
    torch.cuda.synchronize()
    # queues, bit for bit
    rq_t, rq_k = oracle.delay_queues(ev.ev_t, ev.ev_src, ev.ev_n, DT)
    gq_t, gq_k = q.q_t.cpu().numpy(), q.q_k.cpu().numpy()
    for b in range(ev.B):
        k = int(ev.ev_n[b])
        assert np.array_equal(gq_k[b, :, :k], rq_k[b, :, :k]), f"{label}: queue order of sample {b}"
        assert np.array_equal(gq_t[b, :, :k].view(np.uint32), rq_t[b, :, :k].view(np.uint32)), \
            f"{label}: arrival times of sample {b}"
    qs = q.status.cpu().numpy()
    assert qs[0] == 0 and qs[6] == int(ev.ev_n.sum())
    # spikes
    ref = oracle.forward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, WT, DT, OP)
    st = compare_spikes(out.out_t.cpu().numpy(), out.out_n.cpu().numpy(), ref, out.out_i.cpu().numpy(), label=label,
                        out_k_gpu=out.out_k.cpu().numpy())
    status = out.status.cpu().numpy()
    assert status[2] == int(out.out_n.cpu().numpy().sum()) and status[6] == int(ev.ev_n.sum())
    assert not (status[0] & lif.WARN_INTERNAL)
    # the sequential baseline on the same queues
    seq = lif.forward_delayed(q, s, n, w, P, sequential=True)
    torch.cuda.synchronize()
    compare_spikes(seq.out_t.cpu().numpy(), seq.out_n.cpu().numpy(), ref, seq.out_i.cpu().numpy(),
                   label=f"{label} (sequential)", out_k_gpu=seq.out_k.cpu().numpy())
    ss = seq.status.cpu().numpy()
    assert ss[2] == int(seq.out_n.cpu().numpy().sum()) and ss[6] == int(ev.ev_n.sum())
    print(f"    spikes {st['spikes']} flagged {st['flagged']} excused {st['excused']}", flush=True)
    if not grads:
        return st
    # gradients on identical inputs: the oracle's spikes in float32
    rng = np.random.default_rng(5)
    r32 = ref.rounded()
    g = (rng.standard_normal(ref.out_t.shape) * np.isfinite(ref.out_t)).astype(np.float32)
    fwd = lif.ForwardOut(_dev(torch, r32.out_t.astype(np.float32)), _dev(torch, ref.out_n),
                         _dev(torch, r32.out_i.astype(np.float32)), None, _dev(torch, ref.out_k))
    gW, gD, gT = lif.backward_delayed(q, s, n, w, fwd, _dev(torch, g), P)
    torch.cuda.synchronize()
    rW, rD, rT = oracle.backward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, WT, DT, r32, g.astype(np.float64), OP)
    ew = compare_grad(gW.cpu().numpy(), rW, label=f"{label} grad_W")
    ed = compare_grad(gD.cpu().numpy(), rD, label=f"{label} grad_D")
    et = compare_grad(gT.cpu().numpy(), rT, label=f"{label} grad_t")
    assert (gT.cpu().numpy()[np.arange(ev.E_max)[None, :] >= ev.ev_n[:, None]] == 0).all()
    print(f"    rel(gW) {ew:.2e} rel(gD) {ed:.2e} rel(gT) {et:.2e}", flush=True)
    if twice:
        gW2, gD2, gT2 = lif.backward_delayed(q, s, n, w, fwd, _dev(torch, g), P)
        q2 = lif.delay_queues(t, s, n, d)
        out2 = lif.forward_delayed(q2, s, n, w, P)
        for a, b_ in ((gW, gW2), (gD, gD2), (gT, gT2), (out.out_t, out2.out_t)):
            assert torch.equal(a.view(torch.int32), b_.view(torch.int32)), f"{label}: not reproducible"
        k1, k2 = q.q_k.cpu().numpy(), q2.q_k.cpu().numpy()     # entries past ev_n are not written
        for b in range(ev.B):
            assert np.array_equal(k1[b, :, :ev.ev_n[b]], k2[b, :, :ev.ev_n[b]]), f"{label}: queues differ"
    return st


@pytest.mark.parametrize("N", [70, 64, 3])
def test_delays_small_ragged(env, N):
    cfg = W.random_small(81, B=5, C=40, N=N, n_events=600, T=0.5, gain=7.0)
    ev = cfg.events
    ev.ev_n[1] = 0
    run_case(env, ev, cfg.layers[0].WT, W.uniform_delays(81, 40, N), f"ragged N={N}")


def test_delays_reset_and_t_end(env):
    torch, lif = env
    cfg = W.random_small(82, B=3, C=30, N=50, n_events=500, T=0.4, gain=14.0)
    P, OP = lif.Params(v_reset=-0.3, t_end=0.45), oracle.LifParams(v_reset=-0.3, t_end=0.45)
    run_case(env, cfg.events, cfg.layers[0].WT, W.uniform_delays(82, 30, 50, d_max=0.05), "v_reset=-0.3 t_end=0.45",
             P=P, OP=OP)


def test_delays_zero_and_ties(env):
    """Zero delays give the sample's queue (the layer's own spikes), and
    equal arrivals keep the event order."""
    torch, lif = env
    rng = np.random.default_rng(83)
    C, N, n = 16, 40, 400
    t = (rng.integers(0, 64, n) / 128.0).astype(np.float32)          # many equal times
    src = rng.integers(0, C, n).astype(np.int32)
    ev = W.pack_events([t, t[: n // 2]], [src, src[: n // 2]])
    WT = (rng.standard_normal((C, N)) * 5 / math.sqrt(C)).astype(np.float32)
    DT = np.zeros((C, N), np.float32)
    DT[: C // 2] = (rng.integers(0, 4, (C // 2, N)) / 128.0).astype(np.float32)   # equal arrivals across channels
    run_case(env, ev, WT, DT, "ties")
    run_case(env, ev, WT, np.zeros_like(WT), "zero delays", grads=False, twice=False)


def test_delays_spike_cap(env):
    torch, lif = env
    cfg = W.random_small(84, B=2, C=20, N=30, n_events=800, T=0.3, gain=30.0)
    P, OP = lif.Params(s_max=4), oracle.LifParams(s_max=4)
    st = run_case(env, cfg.events, cfg.layers[0].WT, W.uniform_delays(84, 20, 30), "cap s_max=4", P=P, OP=OP,
                  twice=False)
    assert st["spikes"] > 0


def test_bad_delay_reported(env):
    torch, lif = env
    cfg = W.random_small(85, B=2, C=10, N=8, n_events=50, T=0.2, gain=4.0)
    ev = cfg.events
    DT = W.uniform_delays(85, 10, 8)
    DT[3, 5] = -0.01
    q = lif.delay_queues(*(_dev(torch, a) for a in (ev.ev_t, ev.ev_src, ev.ev_n, DT)))
    torch.cuda.synchronize()
    assert q.status.cpu().numpy()[0] & lif.WARN_BAD_DELAY


def test_delays_wide_input(env):
    """More input channels than the LDS column sums of the backward hold
    (C_in > 4096): dL/dW and dL/dD go straight to global memory."""
    cfg = W.random_small(87, B=3, C=4500, N=12, n_events=900, T=0.5, gain=60.0)
    ev = cfg.events
    st = run_case(env, ev, cfg.layers[0].WT, W.uniform_delays(87, 4500, 12), "wide input C_in=4500")
    assert st["spikes"] > 0


@pytest.mark.parametrize("n_events,gain", [(10000, 2.0), (12000, 2.0), (17000, 1.4)])
def test_delays_long_queues(env, n_events, gain):
    """Queues past the 512-thread register/LDS sort (E_max > 8192) take the
    768-thread one up to 11520 and the 1024-thread one up to 16384; past
    16384 they bin through global memory."""
    cfg = W.random_small(86, B=2, C=60, N=20, n_events=n_events, T=2.0 * n_events / 12000, gain=gain)
    ev = cfg.events
    assert ev.E_max > 8192 and (n_events < 16384 or ev.E_max > 16384)
    run_case(env, ev, cfg.layers[0].WT, W.uniform_delays(86, 60, 20), f"long queues E_max={ev.E_max}")


@pytest.mark.timeout(600)
def test_delays_config2_shape(env):
    """The 700 -> 256 layer at B = 32 (~5k events per sample) with the
    paper's delay initialisation U[0, 0.1] s and a gain that makes it fire."""
    cfg = W.config2(gain=6.0)
    run_case(env, cfg.events, cfg.layers[0].WT, W.uniform_delays(2, 700, 256), "config-2 shape, gain 6")


@pytest.mark.parametrize("t_end,vr", [(math.inf, 0.0), (0.5, -0.3)])
def test_delayed_regularisers(env, t_end, vr):
    """Spike-count regularisers of a layer with delays (each neuron's
    intervals between its own arrivals): the hinge means and loss values,
    then the upstream spike-time gradient and the direct weight, delay and
    input-time parts against the oracle on identical inputs (the oracle's
    spike trains in float32), the full gradients through the delayed
    backward, and bitwise reproducibility."""
    from oracle import loss as OL
    from tests.parity import compare_grad_band
    torch, lif = env
    cfg = W.random_small(54, B=4, C=40, N=70, n_events=600, T=0.4, gain=7.0)
    ev, WT = cfg.events, cfg.layers[0].WT
    ev.ev_n[2] = 0
    DT = W.uniform_delays(54, 40, 70, d_max=0.05)
    P = oracle.LifParams(s_max=64, t_end=t_end, v_reset=vr)
    r = oracle.forward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, WT, DT, P)
    assert r.out_n.sum() > 100 and not r.capped.any()
    c_target = float(np.median(r.out_n.mean(axis=0))) + 0.5
    rp = OL.RegParams(c_target=c_target, lam_reg=0.8, lam_over=0.3)
    r32 = r.rounded()
    q_t, q_k = oracle.delay_queues(ev.ev_t, ev.ev_src, ev.ev_n, DT)
    print(f"[case] delayed regularisers t_end={t_end} v_reset={vr} spikes={int(r.out_n.sum())} "
          f"c_target={c_target}", flush=True)
    tables = OL.delayed_interval_tables(ev.ev_src, ev.ev_n, WT, q_t, q_k, r32.out_t, r.out_k, r.out_n, P.tau_mem,
                                        P.tau_syn, P.v_th, P.v_reset, P.t_end)
    under = np.array([[np.mean([max(P.v_th - x[4], 0.0) for x in t if not x[6]] or [0.0]) for t in row]
                      for row in tables])
    over = np.array([[np.mean([max(x[4] - P.v_th, 0.0) for x in t if x[6]] or [0.0]) for t in row]
                     for row in tables])
    L_reg, L_over, gWd, gDd, gTd, gS = OL.spike_count_reg_delayed_grad(
        ev.ev_t, ev.ev_src, ev.ev_n, WT, q_t, q_k, r32.out_t, r.out_k, r.out_n, P.tau_mem, P.tau_syn, P.v_th,
        P.v_reset, P.t_end, rp)
    gWs, gDs, gTs = oracle.backward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, WT, DT, r32, gS, P)
    # the oracle at its exact spike times (the band of the float32 hand-over)
    _, _, hWd, hDd, hTd, hS = OL.spike_count_reg_delayed_grad(
        ev.ev_t, ev.ev_src, ev.ev_n, WT, q_t, q_k, r.out_t, r.out_k, r.out_n, P.tau_mem, P.tau_syn, P.v_th,
        P.v_reset, P.t_end, rp)
    hWs, hDs, hTs = oracle.backward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, WT, DT, r, hS, P)
    t, s, n, w, d = (_dev(torch, a) for a in (ev.ev_t, ev.ev_src, ev.ev_n, WT, DT))
    q = lif.delay_queues(t, s, n, d)
    fwd = lif.ForwardOut(_dev(torch, r32.out_t.astype(np.float32)), _dev(torch, r.out_n),
                         _dev(torch, r32.out_i.astype(np.float32)), None, _dev(torch, r.out_k))
    lp = lif.Params(s_max=64, t_end=t_end, v_reset=vr)
    loss, gu, go = lif.spike_count_reg_delayed(q, s, n, w, fwd, c_target, lp)
    torch.cuda.synchronize()
    for got, ref, label in ((gu.cpu().numpy(), under, "under"), (go.cpu().numpy(), over, "over")):
        err = np.abs(got - ref) - 1e-5 * np.abs(ref)
        assert (err <= 1e-7 * max(np.abs(ref).max(), 1e-30)).all(), label
    assert (gu.cpu().numpy()[2] == P.v_th).all()            # the empty sample: V = 0 throughout
    assert abs(loss[0].item() - L_reg) <= 1e-5 * abs(L_reg)
    assert abs(loss[1].item() - L_over) <= 1e-5 * max(abs(L_over), 1e-12)
    seed = torch.full((ev.B, WT.shape[1], 64), 0.25, device="cuda:0") * fwd.out_t.isfinite()
    loss2, gsp, gW, gD, gT = lif.spike_count_reg_delayed_backward(q, s, n, w, fwd, c_target, 0.8, 0.3, lp,
                                                                  grad_spike=seed.clone())
    torch.cuda.synchronize()
    assert torch.equal(loss.view(torch.int32), loss2.view(torch.int32))
    g_spike = (gsp - seed).cpu().numpy()
    assert np.abs(gS).max() > 0 and np.abs(gWd).max() > 0 and np.abs(gDd).max() > 0
    res = [compare_grad_band(g_spike, gS, hS, label="delayed regulariser spike-time gradient"),
           compare_grad_band(gW.cpu().numpy(), gWd, hWd, label="delayed regulariser direct grad_W"),
           compare_grad_band(gD.cpu().numpy(), gDd, hDd, label="delayed regulariser direct grad_D"),
           compare_grad_band(gT.cpu().numpy(), gTd, hTd, label="delayed regulariser direct grad_t")]
    bW, bD, bT = lif.backward_delayed(q, s, n, w, fwd, gsp - seed, lp)
    torch.cuda.synchronize()
    res += [compare_grad_band((gW + bW).cpu().numpy(), gWd + gWs, hWd + hWs, label="delayed regulariser grad_W"),
            compare_grad_band((gD + bD).cpu().numpy(), gDd + gDs, hDd + hDs, label="delayed regulariser grad_D"),
            compare_grad_band((gT + bT).cpu().numpy(), gTd + gTs, hTd + hTs, label="delayed regulariser grad_t")]
    print("    norm-wise errors (ill-conditioned fractions): spike, direct W D t, full W D t: " +
          ", ".join(f"{e:.1e} ({f:.3f})" for e, f in res), flush=True)
    loss3, gsp3, gW3, gD3, gT3 = lif.spike_count_reg_delayed_backward(q, s, n, w, fwd, c_target, 0.8, 0.3, lp,
                                                                      grad_spike=seed.clone())
    for a, b_ in ((gsp, gsp3), (gW, gW3), (gD, gD3), (gT, gT3)):
        assert torch.equal(a.view(torch.int32), b_.view(torch.int32)), "not reproducible"


def test_delayed_regularisers_wide_input(env):
    """C_in > 4096: the regulariser gradient's dL/dW and dL/dD go straight to
    global memory; direct parts against the oracle."""
    from oracle import loss as OL
    from tests.parity import compare_grad
    torch, lif = env
    cfg = W.random_small(88, B=3, C=4500, N=12, n_events=900, T=0.5, gain=60.0)
    ev, WT = cfg.events, cfg.layers[0].WT
    DT = W.uniform_delays(88, 4500, 12)
    P = oracle.LifParams()
    r = oracle.forward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, WT, DT, P)
    assert r.out_n.sum() > 20
    r32 = r.rounded()
    rp = OL.RegParams(c_target=2.0, lam_reg=0.8, lam_over=0.3)
    q_t, q_k = oracle.delay_queues(ev.ev_t, ev.ev_src, ev.ev_n, DT)
    L_reg, L_over, gWd, gDd, gTd, gS = OL.spike_count_reg_delayed_grad(
        ev.ev_t, ev.ev_src, ev.ev_n, WT, q_t, q_k, r32.out_t, r.out_k, r.out_n, P.tau_mem, P.tau_syn, P.v_th,
        P.v_reset, P.t_end, rp)
    print(f"[case] delayed regularisers C_in=4500 spikes={int(r.out_n.sum())}", flush=True)
    t, s, n, w, d = (_dev(torch, a) for a in (ev.ev_t, ev.ev_src, ev.ev_n, WT, DT))
    q = lif.delay_queues(t, s, n, d)
    fwd = lif.ForwardOut(_dev(torch, r32.out_t.astype(np.float32)), _dev(torch, r.out_n),
                         _dev(torch, r32.out_i.astype(np.float32)), None, _dev(torch, r.out_k))
    loss, gsp, gW, gD, gT = lif.spike_count_reg_delayed_backward(q, s, n, w, fwd, 2.0, 0.8, 0.3, lif.Params())
    torch.cuda.synchronize()
    assert abs(loss[0].item() - L_reg) <= 1e-5 * abs(L_reg)
    compare_grad(gsp.cpu().numpy(), gS, label="wide spike-time gradient")
    compare_grad(gW.cpu().numpy(), gWd, label="wide direct grad_W")
    compare_grad(gD.cpu().numpy(), gDd, label="wide direct grad_D")
    compare_grad(gT.cpu().numpy(), gTd, label="wide direct grad_t")


def test_delayed_regularisers_long_queues(env):
    """E_max > 16384: the per-event dL/dt terms are summed over two ranges of
    event indices; every output against the oracle at the float32 spike
    times (with the hand-over band of the oracle at its exact ones), and
    bitwise reproducible."""
    from oracle import loss as OL
    from tests.parity import compare_grad_band
    torch, lif = env
    cfg = W.random_small(91, B=2, C=60, N=6, n_events=17000, T=2.0 * 17000 / 12000, gain=1.0)
    ev, WT = cfg.events, cfg.layers[0].WT
    assert ev.E_max > 16384
    DT = W.uniform_delays(91, 60, 6)
    P = oracle.LifParams()
    r = oracle.forward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, WT, DT, P)
    assert r.out_n.sum() > 10 and not r.capped.any()
    r32 = r.rounded()
    c_target = float(np.median(r.out_n.mean(axis=0))) + 0.5
    rp = OL.RegParams(c_target=c_target, lam_reg=0.8, lam_over=0.3)
    q_t, q_k = oracle.delay_queues(ev.ev_t, ev.ev_src, ev.ev_n, DT)
    at32, at64 = (OL.spike_count_reg_delayed_grad(ev.ev_t, ev.ev_src, ev.ev_n, WT, q_t, q_k, x.out_t, r.out_k,
                                                  r.out_n, P.tau_mem, P.tau_syn, P.v_th, P.v_reset, P.t_end, rp)
                  for x in (r32, r))
    print(f"[case] delayed regularisers E_max={ev.E_max} spikes={int(r.out_n.sum())}", flush=True)
    t, s, n, w, d = (_dev(torch, a) for a in (ev.ev_t, ev.ev_src, ev.ev_n, WT, DT))
    q = lif.delay_queues(t, s, n, d)
    fwd = lif.ForwardOut(_dev(torch, r32.out_t.astype(np.float32)), _dev(torch, r.out_n),
                         _dev(torch, r32.out_i.astype(np.float32)), None, _dev(torch, r.out_k))
    outs = []
    for _ in range(2):
        loss, gsp, gW, gD, gT = lif.spike_count_reg_delayed_backward(q, s, n, w, fwd, c_target, 0.8, 0.3,
                                                                     lif.Params())
        torch.cuda.synchronize()
        outs.append([x.cpu().numpy() for x in (loss, gsp, gW, gD, gT)])
    loss, gsp, gW, gD, gT = outs[0]
    for i in range(2):                        # L_reg, L_over: inside the band, 1e-5 relative
        lo, hi = sorted((at32[i], at64[i]))
        assert lo - 1e-5 * abs(lo) <= loss[i] <= hi + 1e-5 * abs(hi), (i, loss[i], at32[i], at64[i])
    for got, j, label in ((gsp, 5, "spike-time gradient"), (gW, 2, "direct grad_W"), (gD, 3, "direct grad_D"),
                          (gT, 4, "direct grad_t")):
        compare_grad_band(got, at32[j], at64[j], label=f"long-queue {label}")
    assert (gT[np.arange(ev.E_max)[None, :] >= ev.ev_n[:, None]] == 0).all()
    for a, b_ in zip(outs[0], outs[1]):
        assert np.array_equal(a.view(np.uint32), b_.view(np.uint32)), "not reproducible"
