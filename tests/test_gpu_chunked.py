"""GPU parity of the paper's chunked scheme (lif_layer_forward_chunked)
against the chunk-mode oracle on the same seeded inputs: spikes, and the
consumed and processed event counts of every (sample, neuron) without a
flagged near-tie."""
import numpy as np
import pytest

import oracle
import workloads as W
from tests.parity import compare_spikes

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


def run_case(env, ev, WT, K, C, label, s_max=64):
    torch, lif = env
    print(f"[case] {label} B={ev.B} E_max={ev.E_max} N={WT.shape[1]} K={K} C={C}", flush=True)
    args = [_dev(torch, a) for a in (ev.ev_t, ev.ev_src, ev.ev_n, WT)]
    out, cons, proc = lif.forward_chunked(*args, K=K, C=C, params=lif.Params(s_max=s_max))
    torch.cuda.synchronize()
    Cr = C if C > 0 else (ev.E_max + K - 1) // K + s_max
    ref, rc, rp = oracle.forward_chunked(ev.ev_t, ev.ev_src, ev.ev_n, WT, K, Cr, oracle.LifParams(s_max=s_max))
    s = compare_spikes(out.out_t.cpu().numpy(), out.out_n.cpu().numpy(), ref, out.out_i.cpu().numpy(), label=label,
                       out_k_gpu=out.out_k.cpu().numpy())
    ok = ~np.isfinite(ref.tie_t)
    gc, gp = cons.cpu().numpy(), proc.cpu().numpy()
    assert np.array_equal(gc[ok], rc[ok]), f"{label}: consumed differs"
    assert np.array_equal(gp[ok], rp[ok]), f"{label}: processed differs"
    st = out.status.cpu().numpy()
    assert st[2] == out.out_n.cpu().numpy().sum() and st[6] == int(ev.ev_n.sum())
    assert st[4] == int(gp.astype(np.int64).sum())
    retained = rc.sum() / max(rp.sum(), 1)
    print(f"    spikes {s['spikes']} flagged {s['flagged']} excused {s['excused']} work retained {retained:.3f} "
          f"consumed {rc.sum()}/{int(ev.ev_n.sum()) * WT.shape[1]}", flush=True)
    return gc, gp, rc, rp, ref


@pytest.mark.parametrize("K", [64, 128, 256])
def test_chunked_small_ragged(env, K):
    cfg = W.random_small(71, B=4, C=30, N=70, n_events=700, T=0.5, gain=12.0)
    ev = cfg.events
    ev.ev_n[1] = 0
    gc, gp, rc, rp, ref = run_case(env, ev, cfg.layers[0].WT, K, 10 ** 6, f"ragged K={K}")
    # enough budget: every neuron that is not capped consumes its queue
    full = np.broadcast_to(ev.ev_n[:, None], rc.shape)
    assert (rc[ref.capped == 0] == full[ref.capped == 0]).all() and (ref.capped == 0).any()


@pytest.mark.parametrize("K,C", [(64, 4), (128, 3), (256, 12)])
def test_chunked_budget_runs_out(env, K, C):
    cfg = W.random_small(72, B=3, C=30, N=70, n_events=900, T=0.5, gain=14.0)
    gc, gp, rc, rp, _ = run_case(env, cfg.events, cfg.layers[0].WT, K, C, f"budget K={K} C={C}")
    assert (rc < cfg.events.ev_n[:, None]).any()


def test_chunked_config2_default_budget(env):
    """The 700 -> 256, B = 32 workload at K = 128 with the paper's budget
    rule (ceil(E_max / K) + s_max iterations)."""
    cfg = W.config2()
    run_case(env, cfg.events, cfg.layers[0].WT, 128, 0, "c2 K=128")
