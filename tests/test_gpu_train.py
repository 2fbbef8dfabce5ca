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
    return dict(r1=r1, r2=r2, q2=q2, q3=q3, loss=loss, z=z, gW1=gW1, gW2=gW2, gWo=gWo)


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
