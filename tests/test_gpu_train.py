"""One training step of the two-layer network (paper_2603_13283_amd.train)
on the GPU against the oracle's chain on the same seeded inputs and weights:
input -> LIF -> merge -> LIF -> merge -> weighted LI readout with
temperature cross-entropy, gradients chained back through both merges, and
the Adam update."""
import math

import numpy as np
import pytest

import oracle
import workloads as W
from oracle import loss as OL
from tests.parity import compare_grad, compare_grad_band, compare_spikes

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


def _scatter(gt, perm, n, shape):
    """Queue-time gradient back to the spike slots [B, N, s_max]."""
    B, N, S = shape
    g = np.zeros(shape)
    for b in range(B):
        k = np.arange(int(n[b]))
        p = perm[b, k]
        g[b, p // S, p % S] = gt[b, k]
    return g


def oracle_chain(ev, W1, W2, Wo, labels, OP1, OP2, q, E2, E3):
    r1 = oracle.forward(ev.ev_t, ev.ev_src, ev.ev_n, W1, OP1)
    q2 = oracle.merge(r1.out_t.astype(np.float32), r1.out_n, E2)
    r2 = oracle.forward(q2[0], q2[1], q2[2], W2, OP2)
    q3 = oracle.merge(r2.out_t.astype(np.float32), r2.out_n, E3)
    z = OL.li_readout(q3[0], q3[1], q3[2], Wo, q)
    loss, dz = OL.ce_with_temperature(z, labels, q.beta)
    gWo, gT3 = OL.li_readout_grad(q3[0], q3[1], q3[2], Wo, q, dz)
    g2 = _scatter(gT3.astype(np.float32), q3[3], q3[2], r2.out_t.shape)
    r2_32 = r2.rounded()
    gW2, gT2 = oracle.backward(q2[0], q2[1], q2[2], W2, r2_32, g2, OP2)
    g1 = _scatter(gT2.astype(np.float32), q2[3], q2[2], r1.out_t.shape)
    gW1, _ = oracle.backward(ev.ev_t, ev.ev_src, ev.ev_n, W1, r1.rounded(), g1, OP1)
    return dict(r1=r1, r2=r2, q2=q2, q3=q3, loss=loss, z=z, gW1=gW1, gW2=gW2, gWo=gWo, gT3=gT3)


def _adam(p, g, t, lr, b1, b2, eps):
    """Kingma & Ba's update from zero moments after t identical gradients
    g: m = (1 - b1^t) g, v = (1 - b2^t) g^2 after bias correction give
    m_hat = g, v_hat = g^2."""
    return p - lr * g / (np.abs(g) + eps)


@pytest.mark.timeout(600)
def test_two_layer_training_step(env):
    torch, lif = env
    from paper_2603_13283_amd.train import AdamParams, TwoLayerNet
    C, N1, N2, K, B = 120, 64, 48, 10, 6
    cfg = W.random_small(17, B=B, C=C, N=N1, n_events=900, T=0.5, gain=12.0)
    ev = cfg.events
    rng = np.random.default_rng(18)
    W1 = cfg.layers[0].WT
    W2 = (rng.normal(0, 1, (N1, N2)) * 8.0 / math.sqrt(N1)).astype(np.float32)
    Wo = (rng.normal(0, 1, (N2, K)) * 4.0 / math.sqrt(N2)).astype(np.float32)
    labels = rng.integers(0, K, B).astype(np.int32)
    P1, P2 = lif.Params(s_max=64), lif.Params(s_max=64)
    OP1, OP2 = oracle.LifParams(s_max=64), oracle.LifParams(s_max=64)
    q = OL.LiParams(tau_li=0.5, tau_max=0.6, beta=0.2)
    lq = lif.LiParams(q.tau_mem, q.tau_syn, q.tau_li, q.tau_max, q.beta)
    E2, E3 = 4096, 4096
    print(f"[case] train step B={B} C={C} N1={N1} N2={N2} K={K}", flush=True)
    ref = oracle_chain(ev, W1, W2, Wo, labels, OP1, OP2, q, E2, E3)
    assert ref["r1"].out_n.sum() > 50 and ref["r2"].out_n.sum() > 50, "both layers must fire"
    assert not ref["r1"].capped.any() and not ref["r2"].capped.any()

    dW = [_dev(torch, w) for w in (W1, W2, Wo)]
    net = TwoLayerNet(*dW, B=B, E_max=ev.E_max, P1=P1, P2=P2, q=lq, adam=AdamParams(lr=1e-3), E2_max=E2,
                      E3_max=E3)
    inp = [_dev(torch, a) for a in (ev.ev_t, ev.ev_src, ev.ev_n)]
    lab = _dev(torch, labels)
    res = net.step(*inp, lab, update=False)
    torch.cuda.synchronize()
    # stage by stage: the chains see the same queues where the spikes agree
    s1 = compare_spikes(res.fwd1.out_t.cpu().numpy(), res.fwd1.out_n.cpu().numpy(), ref["r1"],
                        res.fwd1.out_i.cpu().numpy(), label="train l1", out_k_gpu=res.fwd1.out_k.cpu().numpy())
    s2 = compare_spikes(res.fwd2.out_t.cpu().numpy(), res.fwd2.out_n.cpu().numpy(), ref["r2"],
                        res.fwd2.out_i.cpu().numpy(), label="train l2", out_k_gpu=res.fwd2.out_k.cpu().numpy())
    assert s1["flagged"] == 0 and s2["flagged"] == 0, "a near tie would let the chains diverge"
    assert np.array_equal(res.queue3[2].cpu().numpy(), ref["q3"][2])
    assert abs(res.loss.item() - ref["loss"]) <= 1e-5 * abs(ref["loss"])
    for k, name in (("gWo", "Wo"), ("gW2", "W2"), ("gW1", "W1")):
        compare_grad(res.grads[name].cpu().numpy(), ref[k], label=f"train grad {name}")
    # the sequential forward gives the same step
    seq = net.step(*inp, lab, sequential=True, update=False)
    torch.cuda.synchronize()
    assert abs(seq.loss.item() - ref["loss"]) <= 1e-5 * abs(ref["loss"])
    for k, name in (("gWo", "Wo"), ("gW2", "W2"), ("gW1", "W1")):
        compare_grad(seq.grads[name].cpu().numpy(), ref[k], label=f"train grad {name} (sequential forward)")
    # the Adam update (first step: m_hat = g, v_hat = g^2)
    before = [w.cpu().numpy().astype(np.float64) for w in dW]
    res = net.step(*inp, lab, update=True)
    torch.cuda.synchronize()
    for w0, w1, name in zip(before, dW, ("W1", "W2", "Wo")):
        g = res.grads[name].cpu().numpy().astype(np.float64)
        want = _adam(w0, g, 1, 1e-3, 0.9, 0.999, 1e-8)
        assert np.allclose(w1.cpu().numpy(), want, rtol=1e-6, atol=1e-7), name
    print(f"    l1 spikes {s1['spikes']} l2 spikes {s2['spikes']} loss {res.loss.item():.6f} vs {ref['loss']:.6f}",
          flush=True)


def _net_case(seed=17, gain2=8.0):
    C, N1, N2, K, B = 120, 64, 48, 10, 6
    cfg = W.random_small(seed, B=B, C=C, N=N1, n_events=900, T=0.5, gain=12.0)
    rng = np.random.default_rng(seed + 1)
    W1 = cfg.layers[0].WT
    W2 = (rng.normal(0, 1, (N1, N2)) * gain2 / math.sqrt(N1)).astype(np.float32)
    Wo = (rng.normal(0, 1, (N2, K)) * 4.0 / math.sqrt(N2)).astype(np.float32)
    labels = rng.integers(0, K, B).astype(np.int32)
    return cfg.events, W1, W2, Wo, labels, rng


@pytest.mark.timeout(600)
def test_training_step_with_regularisers(env):
    """The step with the spike-count regularisers on both hidden layers (App.
    E.1): each layer's terms weighted by its share of the hidden neurons,
    their spike-time gradients added to the downstream ones before the
    layer's backward, their direct parts added after it."""
    torch, lif = env
    from paper_2603_13283_amd.train import AdamParams, RegConfig, TwoLayerNet
    ev, W1, W2, Wo, labels, _ = _net_case()
    B = ev.B
    OP1, OP2 = oracle.LifParams(s_max=64), oracle.LifParams(s_max=64)
    q = OL.LiParams(tau_li=0.5, tau_max=0.6, beta=0.2)
    E2, E3 = 4096, 4096
    ref = oracle_chain(ev, W1, W2, Wo, labels, OP1, OP2, q, E2, E3)
    r1, r2 = ref["r1"], ref["r2"]
    c1 = float(np.median(r1.out_n.mean(axis=0))) + 0.5
    c2 = float(np.median(r2.out_n.mean(axis=0))) + 0.5
    lam_reg, lam_over = 0.05, 0.02
    n_all = W1.shape[1] + W2.shape[1]
    print(f"[case] train step with regularisers c_target=({c1}, {c2})", flush=True)
    # the oracle's chain with the regulariser terms
    q2, q3 = ref["q2"], ref["q3"]
    r1_32, r2_32 = r1.rounded(), r2.rounded()
    g2 = _scatter(ref["gT3"].astype(np.float32), q3[3], q3[2], r2.out_t.shape)
    rp2 = OL.RegParams(c_target=c2, lam_reg=lam_reg * W2.shape[1] / n_all, lam_over=lam_over * W2.shape[1] / n_all)
    _, _, gW2d, gT2d, gS2 = OL.spike_count_reg_grad(q2[0], q2[1], q2[2], W2, r2_32.out_t, r2.out_k, r2.out_n,
                                                   OP2.tau_mem, OP2.tau_syn, OP2.v_th, OP2.v_reset, OP2.t_end, rp2)
    g2 = (g2 + gS2).astype(np.float32).astype(np.float64)
    gW2, gT2 = oracle.backward(q2[0], q2[1], q2[2], W2, r2_32, g2, OP2)
    gW2, gT2 = gW2 + gW2d, gT2 + gT2d
    g1 = _scatter(gT2.astype(np.float32), q2[3], q2[2], r1.out_t.shape)
    rp1 = OL.RegParams(c_target=c1, lam_reg=lam_reg * W1.shape[1] / n_all, lam_over=lam_over * W1.shape[1] / n_all)
    _, _, gW1d, _, gS1 = OL.spike_count_reg_grad(ev.ev_t, ev.ev_src, ev.ev_n, W1, r1_32.out_t, r1.out_k, r1.out_n,
                                                OP1.tau_mem, OP1.tau_syn, OP1.v_th, OP1.v_reset, OP1.t_end, rp1)
    g1 = (g1 + gS1).astype(np.float32).astype(np.float64)
    gW1, _ = oracle.backward(ev.ev_t, ev.ev_src, ev.ev_n, W1, r1_32, g1, OP1)
    gW1 = gW1 + gW1d
    # the GPU step
    dW = [_dev(torch, w) for w in (W1, W2, Wo)]
    lq = lif.LiParams(q.tau_mem, q.tau_syn, q.tau_li, q.tau_max, q.beta)
    net = TwoLayerNet(*dW, B=B, E_max=ev.E_max, P1=lif.Params(s_max=64), P2=lif.Params(s_max=64), q=lq,
                      adam=AdamParams(lr=1e-3), E2_max=E2, E3_max=E3,
                      reg=RegConfig(c_target=(c1, c2), lam_reg=lam_reg, lam_over=lam_over))
    inp = [_dev(torch, a) for a in (ev.ev_t, ev.ev_src, ev.ev_n)]
    res = net.step(*inp, _dev(torch, labels), update=False)
    torch.cuda.synchronize()
    s1 = compare_spikes(res.fwd1.out_t.cpu().numpy(), res.fwd1.out_n.cpu().numpy(), r1, res.fwd1.out_i.cpu().numpy(),
                        label="reg l1", out_k_gpu=res.fwd1.out_k.cpu().numpy())
    s2 = compare_spikes(res.fwd2.out_t.cpu().numpy(), res.fwd2.out_n.cpu().numpy(), r2, res.fwd2.out_i.cpu().numpy(),
                        label="reg l2", out_k_gpu=res.fwd2.out_k.cpu().numpy())
    assert s1["flagged"] == 0 and s2["flagged"] == 0
    assert abs(res.loss.item() - ref["loss"]) <= 1e-5 * abs(ref["loss"])
    for got, want, name in ((res.grads["Wo"], ref["gWo"], "Wo"), (res.grads["W2"], gW2, "W2"),
                            (res.grads["W1"], gW1, "W1")):
        rel = compare_grad(got.cpu().numpy(), want, label=f"train+reg grad {name}")
        print(f"    grad {name} rel {rel:.2e}", flush=True)
    # the regulariser terms changed the hidden gradients
    assert np.linalg.norm(gW1 - ref["gW1"]) > 1e-3 * np.linalg.norm(gW1)


def _softplus(x, beta):
    z = beta * x.astype(np.float64)
    return ((np.maximum(z, 0.0) + np.log1p(np.exp(-np.abs(z)))) / beta).astype(np.float32)


@pytest.mark.timeout(600)
def test_training_step_with_delays(env):
    """The step with learnable delays on both hidden layers: delays
    softplus(X) with X the raw parameters, per-neuron queues, the delayed
    backward, the gradient back through the softplus, and Adam on W and X."""
    torch, lif = env
    from paper_2603_13283_amd.train import AdamParams, DelayConfig, TwoLayerNet
    ev, W1, W2, Wo, labels, rng = _net_case(23, gain2=4.8)
    B = ev.B
    beta = 5.0
    # raw parameters whose delays lie in [5, 50] ms
    d1 = rng.uniform(0.005, 0.05, W1.shape)
    d2 = rng.uniform(0.005, 0.05, W2.shape)
    X1 = (np.log(np.expm1(beta * d1)) / beta).astype(np.float32)
    X2 = (np.log(np.expm1(beta * d2)) / beta).astype(np.float32)
    D1, D2 = _softplus(X1, beta), _softplus(X2, beta)
    OP = oracle.LifParams(s_max=64)
    q = OL.LiParams(tau_li=0.5, tau_max=0.7, beta=0.2)
    E2, E3 = 4096, 4096
    print(f"[case] train step with delays B={B}", flush=True)
    r1 = oracle.forward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, W1, D1, OP)
    q2 = oracle.merge(r1.out_t.astype(np.float32), r1.out_n, E2)
    r2 = oracle.forward_delayed(q2[0], q2[1], q2[2], W2, D2, OP)
    q3 = oracle.merge(r2.out_t.astype(np.float32), r2.out_n, E3)
    assert r1.out_n.sum() > 50 and r2.out_n.sum() > 50 and not r1.capped.any() and not r2.capped.any()
    z = OL.li_readout(q3[0], q3[1], q3[2], Wo, q)
    loss, dz = OL.ce_with_temperature(z, labels, q.beta)
    gWo, gT3 = OL.li_readout_grad(q3[0], q3[1], q3[2], Wo, q, dz)
    g2 = _scatter(gT3.astype(np.float32), q3[3], q3[2], r2.out_t.shape)
    gW2, gD2, gT2 = oracle.backward_delayed(q2[0], q2[1], q2[2], W2, D2, r2.rounded(), g2, OP)
    g1 = _scatter(gT2.astype(np.float32), q2[3], q2[2], r1.out_t.shape)
    gW1, gD1, _ = oracle.backward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, W1, D1, r1.rounded(), g1, OP)
    sig = lambda x: 1.0 / (1.0 + np.exp(-beta * x.astype(np.float64)))
    gX1, gX2 = gD1 * sig(X1), gD2 * sig(X2)
    # the GPU step
    dW = [_dev(torch, w) for w in (W1, W2, Wo)]
    dX = [_dev(torch, x) for x in (X1, X2)]
    lq = lif.LiParams(q.tau_mem, q.tau_syn, q.tau_li, q.tau_max, q.beta)
    net = TwoLayerNet(*dW, B=B, E_max=ev.E_max, P1=lif.Params(s_max=64), P2=lif.Params(s_max=64), q=lq,
                      adam=AdamParams(lr=1e-3), E2_max=E2, E3_max=E3,
                      delays=DelayConfig(dX[0], dX[1], beta=beta, adam=AdamParams(lr=1e-3)))
    inp = [_dev(torch, a) for a in (ev.ev_t, ev.ev_src, ev.ev_n)]
    lab = _dev(torch, labels)
    res = net.step(*inp, lab, update=False)
    torch.cuda.synchronize()
    assert np.array_equal(res.delays[0].cpu().numpy(), D1) and np.array_equal(res.delays[1].cpu().numpy(), D2)
    s1 = compare_spikes(res.fwd1.out_t.cpu().numpy(), res.fwd1.out_n.cpu().numpy(), r1, res.fwd1.out_i.cpu().numpy(),
                        label="delays l1", out_k_gpu=res.fwd1.out_k.cpu().numpy())
    s2 = compare_spikes(res.fwd2.out_t.cpu().numpy(), res.fwd2.out_n.cpu().numpy(), r2, res.fwd2.out_i.cpu().numpy(),
                        label="delays l2", out_k_gpu=res.fwd2.out_k.cpu().numpy())
    assert s1["flagged"] == 0 and s2["flagged"] == 0
    assert abs(res.loss.item() - loss) <= 1e-5 * abs(loss)
    for k, want in (("Wo", gWo), ("W2", gW2), ("W1", gW1), ("X2", gX2), ("X1", gX1)):
        rel = compare_grad(res.grads[k].cpu().numpy(), want, label=f"train+delays grad {k}")
        print(f"    grad {k} rel {rel:.2e}", flush=True)
    # the sequential forward gives the same step
    seq = net.step(*inp, lab, sequential=True, update=False)
    torch.cuda.synchronize()
    assert abs(seq.loss.item() - loss) <= 1e-5 * abs(loss)
    compare_grad(seq.grads["X1"].cpu().numpy(), gX1, label="train+delays grad X1 (sequential forward)")
    # the update moves the delays' raw parameters with their own Adam
    before = [x.cpu().numpy().astype(np.float64) for x in dX]
    res = net.step(*inp, lab, update=True)
    torch.cuda.synchronize()
    for x0, x1, k in zip(before, dX, ("X1", "X2")):
        g = res.grads[k].cpu().numpy().astype(np.float64)
        assert np.allclose(x1.cpu().numpy(), _adam(x0, g, 1, 1e-3, 0.9, 0.999, 1e-8), rtol=1e-6, atol=1e-7), k


def test_training_step_with_regularisers_and_delays(env):
    """Both options together: learnable delays on both hidden layers and the
    spike-count regularisers of those delayed layers (each neuron's intervals
    between its own arrivals); the regulariser's delay terms join the
    layer's delay gradient before the softplus."""
    torch, lif = env
    from paper_2603_13283_amd.train import AdamParams, DelayConfig, RegConfig, TwoLayerNet
    ev, W1, W2, Wo, labels, rng = _net_case(23, gain2=4.8)
    B = ev.B
    beta = 5.0
    d1 = rng.uniform(0.005, 0.05, W1.shape)
    d2 = rng.uniform(0.005, 0.05, W2.shape)
    X1 = (np.log(np.expm1(beta * d1)) / beta).astype(np.float32)
    X2 = (np.log(np.expm1(beta * d2)) / beta).astype(np.float32)
    D1, D2 = _softplus(X1, beta), _softplus(X2, beta)
    OP = oracle.LifParams(s_max=64)
    q = OL.LiParams(tau_li=0.5, tau_max=0.7, beta=0.2)
    E2, E3 = 4096, 4096
    r1 = oracle.forward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, W1, D1, OP)
    q2 = oracle.merge(r1.out_t.astype(np.float32), r1.out_n, E2)
    r2 = oracle.forward_delayed(q2[0], q2[1], q2[2], W2, D2, OP)
    q3 = oracle.merge(r2.out_t.astype(np.float32), r2.out_n, E3)
    assert r1.out_n.sum() > 50 and r2.out_n.sum() > 50 and not r1.capped.any() and not r2.capped.any()
    c1 = float(np.median(r1.out_n.mean(axis=0))) + 0.5
    c2 = float(np.median(r2.out_n.mean(axis=0))) + 0.5
    lam_reg, lam_over = 0.05, 0.02
    n_all = W1.shape[1] + W2.shape[1]
    print(f"[case] train step with delays and regularisers B={B} c_target=({c1}, {c2})", flush=True)
    z = OL.li_readout(q3[0], q3[1], q3[2], Wo, q)
    loss, dz = OL.ce_with_temperature(z, labels, q.beta)
    gWo, gT3 = OL.li_readout_grad(q3[0], q3[1], q3[2], Wo, q, dz)
    qt2, qk2 = oracle.delay_queues(q2[0], q2[1], q2[2], D2)
    qt1, qk1 = oracle.delay_queues(ev.ev_t, ev.ev_src, ev.ev_n, D1)
    rp2 = OL.RegParams(c_target=c2, lam_reg=lam_reg * W2.shape[1] / n_all, lam_over=lam_over * W2.shape[1] / n_all)
    rp1 = OL.RegParams(c_target=c1, lam_reg=lam_reg * W1.shape[1] / n_all, lam_over=lam_over * W1.shape[1] / n_all)
    sig = lambda x: 1.0 / (1.0 + np.exp(-beta * x.astype(np.float64)))

    def chain(s1, s2):
        """The oracle's backward chain from the hidden spike trains s1, s2
        (float32-rounded, as handed to the GPU, or exact)."""
        g2 = _scatter(gT3.astype(np.float32), q3[3], q3[2], r2.out_t.shape)
        _, _, gW2d, gD2d, gT2d, gS2 = OL.spike_count_reg_delayed_grad(
            q2[0], q2[1], q2[2], W2, qt2, qk2, s2.out_t, r2.out_k, r2.out_n, OP.tau_mem, OP.tau_syn, OP.v_th,
            OP.v_reset, OP.t_end, rp2)
        g2 = (g2 + gS2).astype(np.float32).astype(np.float64)
        gW2, gD2, gT2 = oracle.backward_delayed(q2[0], q2[1], q2[2], W2, D2, s2, g2, OP)
        gW2, gD2, gT2 = gW2 + gW2d, gD2 + gD2d, gT2 + gT2d
        g1 = _scatter(gT2.astype(np.float32), q2[3], q2[2], r1.out_t.shape)
        _, _, gW1d, gD1d, _, gS1 = OL.spike_count_reg_delayed_grad(
            ev.ev_t, ev.ev_src, ev.ev_n, W1, qt1, qk1, s1.out_t, r1.out_k, r1.out_n, OP.tau_mem, OP.tau_syn,
            OP.v_th, OP.v_reset, OP.t_end, rp1)
        g1 = (g1 + gS1).astype(np.float32).astype(np.float64)
        gW1, gD1, _ = oracle.backward_delayed(ev.ev_t, ev.ev_src, ev.ev_n, W1, D1, s1, g1, OP)
        return {"W2": gW2, "W1": gW1 + gW1d, "X2": gD2 * sig(X2), "X1": (gD1 + gD1d) * sig(X1), "D1d": gD1d,
                "D1": gD1 + gD1d}

    ref32, ref64 = chain(r1.rounded(), r2.rounded()), chain(r1, r2)
    # the GPU step
    dW = [_dev(torch, w) for w in (W1, W2, Wo)]
    dX = [_dev(torch, x) for x in (X1, X2)]
    lq = lif.LiParams(q.tau_mem, q.tau_syn, q.tau_li, q.tau_max, q.beta)
    net = TwoLayerNet(*dW, B=B, E_max=ev.E_max, P1=lif.Params(s_max=64), P2=lif.Params(s_max=64), q=lq,
                      adam=AdamParams(lr=1e-3), E2_max=E2, E3_max=E3,
                      reg=RegConfig(c_target=(c1, c2), lam_reg=lam_reg, lam_over=lam_over),
                      delays=DelayConfig(dX[0], dX[1], beta=beta, adam=AdamParams(lr=1e-3)))
    inp = [_dev(torch, a) for a in (ev.ev_t, ev.ev_src, ev.ev_n)]
    res = net.step(*inp, _dev(torch, labels), update=False)
    torch.cuda.synchronize()
    s1 = compare_spikes(res.fwd1.out_t.cpu().numpy(), res.fwd1.out_n.cpu().numpy(), r1, res.fwd1.out_i.cpu().numpy(),
                        label="reg+delays l1", out_k_gpu=res.fwd1.out_k.cpu().numpy())
    s2 = compare_spikes(res.fwd2.out_t.cpu().numpy(), res.fwd2.out_n.cpu().numpy(), r2, res.fwd2.out_i.cpu().numpy(),
                        label="reg+delays l2", out_k_gpu=res.fwd2.out_k.cpu().numpy())
    assert s1["flagged"] == 0 and s2["flagged"] == 0
    assert abs(res.loss.item() - loss) <= 1e-5 * abs(loss)
    assert len(res.reg_losses) == 2
    compare_grad(res.grads["Wo"].cpu().numpy(), gWo, label="train+reg+delays grad Wo")
    for k in ("W2", "W1", "X2", "X1"):
        rel, ill = compare_grad_band(res.grads[k].cpu().numpy(), ref32[k], ref64[k],
                                     label=f"train+reg+delays grad {k}")
        print(f"    grad {k} rel {rel:.2e} (hand-over sensitive {ill:.3f})", flush=True)
    # the regulariser terms changed the delay gradients
    assert np.linalg.norm(ref32["D1d"]) > 1e-3 * np.linalg.norm(ref32["D1"])
