"""GPU forward parity: liblif.so (through the C ABI) against the float64
oracle on identical seeded float32 inputs."""
import math

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


GPU_ONLY = ("validate", "pool_cap", "root_general")     # options of the GPU path alone


def run_both(env, ev, WT, s_max=64, sequential=False, **kw):
    torch, lif = env
    P = lif.Params(s_max=s_max, **kw)
    OP = oracle.LifParams(s_max=s_max, **{k: v for k, v in kw.items() if k not in GPU_ONLY})
    out = lif.forward(_dev(torch, ev.ev_t), _dev(torch, ev.ev_src), _dev(torch, ev.ev_n), _dev(torch, WT), P,
                      sequential=sequential)
    torch.cuda.synchronize()
    ref = oracle.forward(ev.ev_t, ev.ev_src, ev.ev_n, WT, OP)
    return out, ref


def check(env, ev, WT, label, s_max=64, both=True, **kw):
    print(f"[case] {label} B={ev.B} E_max={ev.E_max} C={WT.shape[0]} N={WT.shape[1]}", flush=True)
    stats = {}
    for seq in ((False, True) if both else (False,)):
        out, ref = run_both(env, ev, WT, s_max=s_max, sequential=seq, **kw)
        st = out.status.cpu().numpy()
        s = compare_spikes(out.out_t.cpu().numpy(), out.out_n.cpu().numpy(), ref, out.out_i.cpu().numpy(),
                           label=f"{label}{' seq' if seq else ''}", out_k_gpu=out.out_k.cpu().numpy())
        assert not st[0] & 64, "internal error flagged by the library"
        assert st[2] == out.out_n.cpu().numpy().sum()
        assert st[6] == int(ev.ev_n.sum())
        assert st[1] == int(ref.capped.sum())
        s["status"] = st.tolist()
        stats["seq" if seq else "par"] = s
    print(f"    {stats}", flush=True)
    return stats


def test_config1_silent_and_driven(env):
    cfg = W.config1()
    s = check(env, cfg.events, cfg.layers[0].WT, "c1")
    assert s["par"]["spikes"] == 0
    cfgd = W.config1(gain=30.0)
    s = check(env, cfgd.events, cfgd.layers[0].WT, "c1x10")
    assert s["par"]["spikes"] > 100


@pytest.mark.parametrize("seed,N", [(1, 64), (2, 70), (3, 20), (4, 200)])
def test_small_ragged(env, seed, N):
    cfg = W.random_small(seed, B=5, C=30, N=N, n_events=700, T=0.5, gain=14.0)
    assert (cfg.events.ev_n == 0).any() or cfg.events.ev_n.min() < cfg.events.E_max
    s = check(env, cfg.events, cfg.layers[0].WT, f"small{seed}")
    assert s["par"]["spikes"] > 20


def test_empty_inputs(env):
    ev = W.pack_events([np.array([]), np.array([])], [np.array([], int), np.array([], int)], e_max=3)
    WT = np.ones((4, 5), np.float32)
    s = check(env, ev, WT, "empty")
    assert s["par"]["spikes"] == 0
    ev1 = W.pack_events([np.array([0.1])], [np.array([2])])
    WT1 = np.full((4, 3), 50.0, np.float32)
    s = check(env, ev1, WT1, "one-event")
    assert s["par"]["spikes"] > 3


def test_equal_times_and_exact_boundaries(env):
    rng = np.random.default_rng(5)
    t = np.sort(np.repeat(rng.random(150) * 0.2, 3))            # every time three times
    src = rng.integers(0, 12, t.size)
    ev = W.pack_events([t], [src])
    WT = (rng.standard_normal((12, 66)) * 3.0).astype(np.float32)
    s = check(env, ev, WT, "dup-times")
    assert s["par"]["spikes"] > 10


def test_reset_nonzero_threshold_and_t_end(env):
    cfg = W.random_small(6, B=3, C=30, N=100, n_events=500, T=0.4, gain=14.0)
    check(env, cfg.events, cfg.layers[0].WT, "vr", v_reset=-0.25)
    check(env, cfg.events, cfg.layers[0].WT, "th0.5", v_th=0.5)
    check(env, cfg.events, cfg.layers[0].WT, "tend", t_end=0.3)
    check(env, cfg.events, cfg.layers[0].WT, "taus", tau_mem=0.03, tau_syn=0.002)


def test_spike_cap(env):
    cfg = W.random_small(7, B=3, C=30, N=100, n_events=500, T=0.4, gain=20.0)
    s = check(env, cfg.events, cfg.layers[0].WT, "cap1", s_max=1)
    assert s["par"]["status"][1] > 0 and s["par"]["status"][0] & 1
    check(env, cfg.events, cfg.layers[0].WT, "cap3", s_max=3)


def test_long_stream_chunks_and_cap(env):
    """Streams of 20 000 events per sample: the resolve pass takes the
    flagged sub-blocks in chunks of 8192 events, so spike chains (up to about
    600 spikes per neuron, flushed 64 at a time) run across window and chunk
    boundaries; with a small cap, neurons stop in an early chunk while later
    chunks of the same sample follow, and with a cap of 100 they stop in a
    later one."""
    cfg = W.random_small(35, B=2, C=40, N=96, n_events=20000, T=4.0, gain=3.0, ragged=False)
    s = check(env, cfg.events, cfg.layers[0].WT, "long", s_max=640, both=False)
    assert s["par"]["spikes"] > 10000 and s["par"]["status"][1] == 0
    s = check(env, cfg.events, cfg.layers[0].WT, "long_cap2", s_max=2, both=False)
    assert s["par"]["status"][1] > 0
    s = check(env, cfg.events, cfg.layers[0].WT, "long_cap100", s_max=100, both=False)
    assert s["par"]["status"][1] > 0


def test_config2_full(env):
    cfg = W.config2()
    s = check(env, cfg.events, cfg.layers[0].WT, "c2")
    assert s["par"]["spikes"] > 100
    assert s["par"]["status"][1] == 0              # the cap never binds


def test_config2_driven(env):
    cfg = W.config2(B=8)
    s = check(env, cfg.events, cfg.layers[0].WT, "c2-th0.5", v_th=0.5)
    assert s["par"]["spikes"] > 1000


def test_config4_bursts_full(env):
    """2312 -> 1024, batch 64, ~20k events per sample in three bursts."""
    cfg = W.config4()
    s = check(env, cfg.events, cfg.layers[0].WT, "c4")
    assert s["par"]["spikes"] > 10000
    assert s["par"]["status"][1] == 0


def test_config5_full_stated_gain(env):
    """32768 -> 2048 at the stated gain, batch 16, ~100k events per sample:
    the hidden layer stays silent on both sides (the driven variant is in
    the two-layer tests)."""
    cfg = W.config5()
    s = check(env, cfg.events, cfg.layers[0].WT, "c5-hidden", both=False)
    assert s["par"]["spikes"] == 0 and s["par"]["status"][6] == int(cfg.events.ev_n.sum())


def test_determinism(env):
    torch, lif = env
    cfg = W.random_small(8, B=4, C=30, N=130, n_events=900, T=0.5, gain=14.0)
    ev, WT = cfg.events, cfg.layers[0].WT
    a = lif.forward(_dev(torch, ev.ev_t), _dev(torch, ev.ev_src), _dev(torch, ev.ev_n), _dev(torch, WT))
    b = lif.forward(_dev(torch, ev.ev_t), _dev(torch, ev.ev_src), _dev(torch, ev.ev_n), _dev(torch, WT))
    torch.cuda.synchronize()
    assert torch.equal(a.out_t, b.out_t) and torch.equal(a.out_n, b.out_n) and torch.equal(a.out_i, b.out_i)
    assert torch.equal(a.out_k, b.out_k)


def test_graph_replay_matches_eager(env):
    """The forward call captured in a HIP graph and replayed several times,
    with other eager forwards (different inputs) and synchronisations
    between the replays, reproduces the eager result every time."""
    torch, lif = env
    cfg = W.random_small(12, B=4, C=40, N=150, n_events=1200, T=0.6, gain=14.0)
    other = W.random_small(13, B=2, C=40, N=150, n_events=700, T=0.6, gain=14.0)
    ev, WT = cfg.events, cfg.layers[0].WT
    d = [_dev(torch, a) for a in (ev.ev_t, ev.ev_src, ev.ev_n, WT)]
    do = [_dev(torch, a) for a in (other.events.ev_t, other.events.ev_src, other.events.ev_n, other.layers[0].WT)]
    P = lif.Params()
    ref = lif.forward(*d, P)
    torch.cuda.synchronize()
    B, E = ev.ev_t.shape
    ws = torch.empty(lif.lif_layer_forward_workspace_size(B, E, WT.shape[0], WT.shape[1], P.c()),
                     dtype=torch.uint8, device="cuda:0")
    out = lif.forward(*d, P, ws=ws)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        lif.forward(*d, P, ws=ws, out=out)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        lif.forward(*d, P, ws=ws, out=out)
    for rep in range(4):
        out.out_t.fill_(-1.0)
        out.out_n.fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.out_t, ref.out_t), rep
        assert torch.equal(out.out_n, ref.out_n), rep
        assert torch.equal(out.out_i, ref.out_i), rep
        assert torch.equal(out.out_k, ref.out_k), rep
        assert torch.equal(out.status, ref.status), rep
        lif.forward(*do, P)                  # eager work between replays
        torch.cuda.synchronize()


def test_validation_flags(env):
    torch, lif = env
    ev = W.pack_events([np.array([0.1, 0.2, 0.3])], [np.array([0, 1, 2])])
    ev.ev_t[0, 1] = 0.5                      # unsorted
    ev.ev_src[0, 2] = 9                      # out of range for C_in = 4
    WT = np.ones((4, 8), np.float32)
    out = lif.forward(_dev(torch, ev.ev_t), _dev(torch, ev.ev_src), _dev(torch, ev.ev_n),
                      _dev(torch, WT), lif.Params(validate=True))
    torch.cuda.synchronize()
    st = out.status.cpu().numpy()
    assert st[0] & lif.WARN_UNSORTED and st[0] & lif.WARN_BAD_SOURCE


def test_record_pool_fallback(env):
    """With a tiny pool of entering states (lif_params.pool_cap) the
    overflowing sub-blocks are rebuilt from the segment's carried state; the
    results match the oracle and are bit-identical to the default pool's."""
    torch, lif = env
    cfg = W.random_small(9, B=3, C=30, N=130, n_events=600, T=0.4, gain=14.0)
    s = check(env, cfg.events, cfg.layers[0].WT, "pool5", both=False, pool_cap=5)
    assert s["par"]["status"][7] > 0
    s = check(env, cfg.events, cfg.layers[0].WT, "pool0", both=False, pool_cap=0)
    assert s["par"]["status"][7] >= s["par"]["status"][4] > 0   # every walked block fell back
    ev = cfg.events
    args = [_dev(torch, a) for a in (ev.ev_t, ev.ev_src, ev.ev_n, cfg.layers[0].WT)]
    outs = [lif.forward(*args, lif.Params(pool_cap=pc)) for pc in (-1, 5, 0)]
    torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(o.out_n, outs[0].out_n) and torch.equal(o.out_k, outs[0].out_k)
        assert torch.equal(o.out_t.view(torch.int32), outs[0].out_t.view(torch.int32))
        assert torch.equal(o.out_i.view(torch.int32), outs[0].out_i.view(torch.int32))


@pytest.mark.parametrize("N", [264, 266, 265])
def test_neurons_per_lane_variants(env, N):
    """The segment walks hold 4, 2 or 1 adjacent neurons per lane, as the
    W^T row length allows (N = 264, 266, 265); every variant matches the
    oracle, and in each the last tile of neurons is partial."""
    npl = 4 if N % 4 == 0 else (2 if N % 2 == 0 else 1)
    cfg = W.random_small(31, B=2, C=50, N=N, n_events=700, T=0.35, gain=12.0)
    s = check(env, cfg.events, cfg.layers[0].WT, f"npl{npl}", both=False)
    assert s["par"]["spikes"] > 0


def test_odd_neuron_count(env):
    """An odd N forces one neuron per lane (no vector weight loads)."""
    cfg = W.random_small(32, B=2, C=40, N=77, n_events=500, T=0.3, gain=12.0)
    s = check(env, cfg.events, cfg.layers[0].WT, "odd-N", both=False)
    assert s["par"]["spikes"] > 0


@pytest.mark.parametrize("general", [False, True])
def test_spike_solver_paths(env, general):
    """tau_m / tau_s = 4 takes the polynomial spike-time solve; the
    LIF_ROOT_GENERAL flag forces the exponential Newton solve on the same
    bursting input (several spikes per interval).  Both match the oracle."""
    cfg = W.random_small(33, B=2, C=30, N=96, n_events=600, T=0.3, gain=20.0)
    s = check(env, cfg.events, cfg.layers[0].WT, f"solver-{'general' if general else 'poly'}", root_general=general)
    assert s["par"]["spikes"] > 50


@pytest.mark.parametrize("ratio", [2.0, 3.0, 3.7, 5.0])
def test_tau_ratios(env, ratio):
    """tau_m / tau_s = 2, 3 and 5 take the polynomial solve with p = 1, 2, 4;
    3.7 takes the exponential solve."""
    cfg = W.random_small(34, B=2, C=30, N=70, n_events=500, T=0.3, gain=16.0)
    s = check(env, cfg.events, cfg.layers[0].WT, f"ratio{ratio}", both=False, tau_mem=0.02, tau_syn=0.02 / ratio)
    assert s["par"]["spikes"] > 0
