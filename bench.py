"""Benchmark of the event-driven LIF layer forward pass on one MI355X.

Workload: one LIF layer, 700 input channels -> 256 neurons, batch 32, 1 s per
sample, lognormal-rate Poisson input channels (~5k events per sample),
W ~ N(0,1) * 4/sqrt(700), tau_m = 20 ms, tau_s = 5 ms, threshold 1, hard
reset to 0 (synthetic, seeded).  A step is one forward pass of the layer
(decays, weight gather, segment scan, interval checks, root solves, resets,
outputs) over the batch, with all inputs resident in HBM.

Prints one JSON line: throughput in neuron-events/s (N_out * sum of events
per sample, per second); the roofline of the forward pass (its algorithmic
bytes over its duration, timed with HIP events on the launch stream, against
the HBM peak); the speedup over the sequential one-thread-per-neuron GPU
event loop; the backward time; the same figures for the other workloads
(two-layer, event-camera and large shapes) as extra keys; and the float64
CPU oracle timed on the host cores on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0     # MI355X HBM3E, GB/s
FORWARD_KERNELS = ("aggregate", "carry", "check", "resolve")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_forward_700x256_b32.txt")
L2_FILE = os.path.join(ROOT, "profiles", "l2_forward_700x256_b32.txt")
KERNEL_SOURCES = ("lif_forward.hip", "lif_common.hpp", "lif_host.hpp", "lif_walk.hpp")


def kernel_sources_sha256() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2603_13283_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def _profile_table(path):
    """Rows `kernel a b` of a profile summary in profiles/, or None when it
    is missing or was taken on other kernel sources than the ones built now."""
    try:
        lines = open(path).read().splitlines()
    except OSError:
        return None
    sha, rows = None, {}
    for ln in lines:
        if ln.startswith("sources_sha256:"):
            sha = ln.split(":", 1)[1].strip()
            continue
        parts = ln.split()
        if not ln.startswith("#") and len(parts) == 3:
            rows[parts[0]] = (float(parts[1]), float(parts[2]))
    if sha != kernel_sources_sha256():
        return None
    return rows


def measured_traffic():
    """HBM bytes of one forward pass (all its kernels) from the rocprofv3
    FETCH_SIZE and WRITE_SIZE runs summarised in profiles/ (already scaled by
    the copy-probe factors), with the per-kernel split, or (None, None)."""
    rows = _profile_table(TRAFFIC_FILE)
    if not rows or not all(k in rows for k in FORWARD_KERNELS):
        return None, None
    per = {k: int(rows[k][0] + rows[k][1]) for k in FORWARD_KERNELS}
    return sum(per.values()), per


def measured_l2():
    """L2 (TCC) hit rate per forward kernel from profiles/, or None."""
    rows = _profile_table(L2_FILE)
    if not rows:
        return None
    return {k: (h / (h + m) if h + m > 0 else None) for k, (h, m) in rows.items()}


def fwd_alg_bytes(total_ev, N, B, spikes):
    """Algorithmic bytes of one forward pass: per event its time and source
    (8 B) and one float32 weight per neuron (4 B per neuron-event); the spike
    counts (4 B per neuron); the spike time and I at each spike (8 B)."""
    return total_ev * (8 + 4 * N) + B * N * 4 + spikes * 8


class Dev:
    def __init__(self, torch, dev):
        self.torch, self.dev = torch, dev

    def __call__(self, a):
        return self.torch.from_numpy(np.ascontiguousarray(a)).to(self.dev)


def time_steps(torch, fn, steps, warmup):
    """Warm up, then time `steps` calls twice: a plain loop by wall clock
    (bracketed by device synchronisations, nothing else enqueued between
    the calls), then a loop with HIP events around every call on the current
    stream (the library launches on it) for per-step statistics.  Returns
    (ms per step by wall clock, per-step event durations in ms)."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps * 1e3
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for a, b in ev:
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    return wall, [a.elapsed_time(b) for a, b in ev]


def stats_ms(xs):
    return {"mean": statistics.fmean(xs), "median": statistics.median(xs),
            "stdev": statistics.stdev(xs) if len(xs) > 1 else 0.0, "min": min(xs), "max": max(xs)}


def run_workload(torch, lif, d, name, ev, WT, P, steps, warmup, seq_steps, backward=False):
    """Forward (and optionally backward) timing of one workload, with the
    sequential GPU loop on the same inputs."""
    B, E = ev.ev_t.shape
    C, N = WT.shape
    total_ev = int(ev.ev_n.sum())
    dt, ds, dn, dW = d(ev.ev_t), d(ev.ev_src), d(ev.ev_n), d(WT)
    pc = P.c()
    ws = torch.empty(lif.lif_layer_forward_workspace_size(B, E, C, N, pc), dtype=torch.uint8, device=d.dev)
    out = lif.forward(dt, ds, dn, dW, P, ws=ws)
    wall, evs = time_steps(torch, lambda: lif.forward(dt, ds, dn, dW, P, ws=ws, out=out), steps, warmup)
    spikes = int(out.out_n.sum().item())
    status = out.status.cpu().numpy().tolist()
    seq = lif.forward(dt, ds, dn, dW, P, sequential=True, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(seq.out_n, out.out_n), f"{name}: sequential and parallel spike counts differ"
    seq_wall, _ = time_steps(torch, lambda: lif.forward(dt, ds, dn, dW, P, sequential=True, ws=ws, out=seq),
                             seq_steps, 0)
    r = {"workload": name, "batch": B, "c_in": C, "n_out": N, "events": total_ev, "e_max": E,
         "neuron_events": N * total_ev, "spikes": spikes, "forward_ms": wall,
         "forward_event_ms": stats_ms(evs), "neuron_events_per_s": N * total_ev / (wall * 1e-3),
         "hbm_frac": fwd_alg_bytes(total_ev, N, B, spikes) / (wall * 1e-3) / 1e9 / HBM_PEAK_GBS,
         "sequential_ms": seq_wall, "speedup_vs_sequential": seq_wall / wall, "status": status,
         "workspace_bytes": int(ws.numel())}
    if backward:
        rng = np.random.default_rng(1)
        valid = np.isfinite(out.out_t.cpu().numpy())
        g = d((rng.standard_normal(valid.shape) * valid).astype(np.float32))
        bws = torch.empty(lif.lif_layer_backward_workspace_size(B, E, C, N, pc), dtype=torch.uint8, device=d.dev)
        bwall, bevs = time_steps(torch, lambda: lif.backward(dt, ds, dn, dW, out, g, P, ws=bws),
                                 max(3, steps // 2), 2)
        r["backward_ms"] = bwall
        r["backward_event_ms"] = stats_ms(bevs)
    log(f"[bench] {name}: forward {wall * 1e3:.1f} us ({r['neuron_events_per_s']:.3e} neuron-events/s, "
        f"{r['hbm_frac']:.1%} of HBM peak), sequential {seq_wall:.3f} ms ({r['speedup_vs_sequential']:.1f}x)"
        + (f", backward {r['backward_ms'] * 1e3:.1f} us" if backward else "") + f", {spikes} spikes")
    del ws
    return r


def train_step(torch, lif, d, c3, steps, warmup, variant="plain"):
    """The paper's training step (two LIF layers, merges, weighted LI readout
    with temperature cross-entropy, backward through both merges, Adam) at
    config 3's shape with a 512 -> 20 readout, with the parallel layers and
    with the sequential baseline in their place.  variant "reg" adds the
    spike-count regularisers to both hidden layers (targets 14, lambda_reg
    1e-3, lambda_over 5e-5, as the paper's SHD model), "delays" learnable
    delays on both hidden layers (initial delays U[0, 0.1) s, softplus
    sharpness 5), "reg_delays" both."""
    from paper_2603_13283_amd.train import AdamParams, DelayConfig, RegConfig, TwoLayerNet
    ev = c3.events
    rng = np.random.default_rng(11)
    Wo = (rng.normal(0, 1, (512, 20)) * 4.0 / np.sqrt(512)).astype(np.float32)
    labels = d(rng.integers(0, 20, ev.B).astype(np.int32))
    inp = [d(ev.ev_t), d(ev.ev_src), d(ev.ev_n)]
    extra = {"plain": "", "reg": " + spike-count regularisers on both hidden layers",
             "delays": " + learnable delays on both hidden layers",
             "reg_delays": " + learnable delays and spike-count regularisers on both hidden layers"}[variant]
    out = {"workload": "700->512->512 LIF + 512->20 weighted LI readout, B=128, ~10k events; forward, "
                       "cross-entropy, backward through both merges, Adam on all parameters" + extra}
    beta = 5.0
    raw = lambda shape: d((np.log(np.expm1(beta * rng.uniform(1e-3, 0.1, shape))) / beta).astype(np.float32))
    for name, seq in (("parallel", False), ("sequential", True)):
        kw = {}
        if variant in ("reg", "reg_delays"):
            kw["reg"] = RegConfig(c_target=(14.0, 14.0), lam_reg=1e-3, lam_over=5e-5)
        if variant in ("delays", "reg_delays"):
            kw["delays"] = DelayConfig(raw((700, 512)), raw((512, 512)), beta=beta, adam=AdamParams(lr=1e-3))
        net = TwoLayerNet(d(c3.layers[0].WT), d(c3.layers[1].WT), d(Wo), B=ev.B, E_max=ev.E_max,
                          P1=lif.Params(s_max=128), P2=lif.Params(s_max=128),
                          q=lif.LiParams(tau_li=0.5, tau_max=1.0, beta=0.05), adam=AdamParams(lr=1e-3), **kw)
        r = net.step(*inp, labels, sequential=seq)
        torch.cuda.synchronize()
        ms, ev_ms = time_steps(torch, lambda: net.step(*inp, labels, sequential=seq), steps if not seq else 3,
                               warmup if not seq else 1)
        out[f"{name}_ms"] = ms
        out[f"{name}_event_ms"] = stats_ms(ev_ms)
        if not seq:
            out["spikes_layer1"] = int(r.fwd1.out_n.sum().item())
            out["spikes_layer2"] = int(r.fwd2.out_n.sum().item())
            out["loss_first_step"] = float(r.loss.item())
        del net, r
    out["speedup_vs_sequential"] = out["sequential_ms"] / out["parallel_ms"]
    log(f"[bench] training step{extra}: {out['parallel_ms']:.2f} ms parallel, {out['sequential_ms']:.2f} ms with "
        f"the sequential layers ({out['speedup_vs_sequential']:.1f}x)")
    return out


def chunk_study(torch, lif, d, ev, WT, steps, warmup, seq_ms):
    """The paper's chunked scheme on the headline workload at chunk sizes 64,
    128 and 256 with its budget rule: time per forward, work retained
    (consumed / processed events) and speedup over the sequential loop."""
    args = [d(ev.ev_t), d(ev.ev_src), d(ev.ev_n), d(WT)]
    out = {"workload": "700->256, B=32, chunked forward (one wave per neuron, K events per iteration, "
                       "budget ceil(E_max/K) + s_max iterations)"}
    for K in (64, 128, 256):
        run = lambda: lif.forward_chunked(*args, K=K, C=0)
        o, cons, proc = run()
        torch.cuda.synchronize()
        ms, ev_ms = time_steps(torch, run, steps, warmup)
        c, p = int(cons.sum().item()), int(proc.sum().item())
        out[f"K{K}"] = {"ms": ms, "event_ms": stats_ms(ev_ms), "work_retained": c / max(p, 1),
                        "consumed": c, "processed": p, "spikes": int(o.out_n.sum().item()),
                        "speedup_vs_sequential": seq_ms / ms}
        log(f"[bench] chunked K={K}: {ms * 1e3:.1f} us, work retained {c / max(p, 1):.3f}, "
            f"{seq_ms / ms:.1f}x the sequential loop")
    return out


def delay_study(torch, lif, d, ev, WT, steps, warmup, seq_steps):
    """The layer with synaptic delays on the headline workload, delays drawn
    U[0, 0.1) s (the paper's initialisation): queue build, forward (one wave
    per neuron on its own queue), the sequential loop on the same queues, and
    the backward (weights, delays, input times)."""
    import workloads as W
    C, N = WT.shape
    DT = W.uniform_delays(2, C, N)
    dt, ds, dn, dW, dD = d(ev.ev_t), d(ev.ev_src), d(ev.ev_n), d(WT), d(DT)
    P = lif.Params(s_max=64)
    qws = torch.empty(lif.lif_delay_queues_workspace_size(ev.B, ev.E_max, N), dtype=torch.uint8, device=dt.device)
    q = lif.delay_queues(dt, ds, dn, dD, ws=qws)
    q_ms, q_ev = time_steps(torch, lambda: lif.delay_queues(dt, ds, dn, dD, ws=qws), steps, warmup)
    fwd = lambda: lif.forward_delayed(q, ds, dn, dW, P)
    o = fwd()
    torch.cuda.synchronize()
    f_ms, f_ev = time_steps(torch, fwd, steps, warmup)
    s_ms, _ = time_steps(torch, lambda: lif.forward_delayed(q, ds, dn, dW, P, sequential=True), seq_steps, 1)
    g = torch.randn(o.out_t.shape, device=dt.device) * torch.isfinite(o.out_t)
    bws = torch.empty(lif.lif_layer_backward_delayed_workspace_size(ev.B, ev.E_max, C, N, P.c()), dtype=torch.uint8,
                      device=dt.device)
    b_ms, b_ev = time_steps(torch, lambda: lif.backward_delayed(q, ds, dn, dW, o, g, P, ws=bws), steps, warmup)
    ne = int(ev.ev_n.sum()) * N
    spikes = int(o.out_n.sum().item())
    log(f"[bench] delays: queues {q_ms * 1e3:.1f} us, forward {f_ms * 1e3:.1f} us ({ne / (f_ms * 1e-3):.3e} "
        f"neuron-events/s), sequential {s_ms:.3f} ms ({s_ms / f_ms:.1f}x), backward {b_ms * 1e3:.1f} us, "
        f"{spikes} spikes")
    return {"workload": "700->256, B=32, ~5k events, delays U[0, 0.1) s: per-neuron queues, forward, backward",
            "queues_ms": q_ms, "queues_event_ms": stats_ms(q_ev), "forward_ms": f_ms, "forward_event_ms": stats_ms(f_ev),
            "neuron_events_per_s": ne / (f_ms * 1e-3), "sequential_ms": s_ms, "speedup_vs_sequential": s_ms / f_ms,
            "backward_ms": b_ms, "backward_event_ms": stats_ms(b_ev), "spikes": spikes}


def cpu_oracle(ev, WT, nthreads, seconds, n_samples, n_neurons):
    """The float64 oracle on a bounded sample of a workload (the first
    n_samples samples and n_neurons neurons), repeated for about `seconds`;
    returns (neuron-events per second, seconds per call, repetitions)."""
    import oracle
    OP = oracle.LifParams(s_max=64)
    sub = np.ascontiguousarray(WT[:, :n_neurons])
    args = (ev.ev_t[:n_samples], ev.ev_src[:n_samples], ev.ev_n[:n_samples], sub, OP)
    oracle.forward(*args, nthreads=nthreads)
    reps = 0
    c0 = time.perf_counter()
    while reps < 2 or time.perf_counter() - c0 < seconds:
        oracle.forward(*args, nthreads=nthreads)
        reps += 1
    per = (time.perf_counter() - c0) / reps
    ne = int(ev.ev_n[:n_samples].sum()) * sub.shape[1]
    return ne / per, per, reps


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--seq-steps", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true", help="time the headline workload only")
    ap.add_argument("--extras", default="", metavar="NAMES",
                    help="comma-separated subset of the other workloads (keys of other_workloads); default all")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="CPU oracle baseline: repeat the bounded sample until this much time has passed")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run one plain device-to-device copy of BYTES bytes (calibrates the HBM byte "
                         "counters of a profiler against a kernel of known traffic) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the layer shards over samples "
              "with no exchange in the forward pass, and multi-GPU runs are not part of this build.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2603_13283_amd as lif
    import workloads as W

    dev = torch.device("cuda:0")
    if args.copy_probe:
        n = args.copy_probe // 4
        a = torch.ones(n, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        log(f"[bench] copy probe: {n * 4} bytes read, {n * 4} bytes written")
        return
    d = Dev(torch, dev)
    cfg = W.config2()
    ev, WT = cfg.events, cfg.layers[0].WT
    B, E = ev.ev_t.shape
    C, N = WT.shape
    total_ev = int(ev.ev_n.sum())
    neuron_events = N * total_ev
    P = lif.Params(s_max=64)
    d_t, d_s, d_n, d_W = d(ev.ev_t), d(ev.ev_src), d(ev.ev_n), d(WT)
    pc = P.c()
    ws = torch.empty(lif.lif_layer_forward_workspace_size(B, E, C, N, pc), dtype=torch.uint8, device=dev)
    out = lif.forward(d_t, d_s, d_n, d_W, P, ws=ws)
    torch.cuda.synchronize()
    log(f"[bench] {cfg.name}: B={B} E_max={E} events={total_ev} N={N} neuron-events={neuron_events} "
        f"lib={lif.lif_version()}")
    fwd = lambda: lif.forward(d_t, d_s, d_n, d_W, P, ws=ws, out=out)

    # ---- per-kernel durations: every launch bracketed by HIP events that
    # its own dispatch records (the library's kernel timer)
    lif.lif_timer_enable(True)
    for _ in range(args.warmup):
        fwd()
    torch.cuda.synchronize()
    lif.lif_timer_enable(True)
    for _ in range(args.steps):
        fwd()
    torch.cuda.synchronize()
    kern = lif.lif_timer_read()
    lif.lif_timer_enable(False)
    kern_us = {k: v[0] / v[1] * 1e3 for k, v in kern.items()}
    log("[bench] kernels: " + ", ".join(f"{k}={v:.1f}us" for k, v in kern_us.items()))

    # ---- the timed steps: eager forward calls
    ms_step, ev_ms = time_steps(torch, fwd, args.steps, args.warmup)
    fst = stats_ms(ev_ms)
    ref_t, ref_n, ref_st = out.out_t.clone(), out.out_n.clone(), out.status.clone()
    value = neuron_events / (ms_step * 1e-3)
    status = out.status.cpu().numpy().tolist()
    n_spikes = int(out.out_n.sum().item())

    # ---- the same call captured once in a HIP graph and replayed
    gstream = torch.cuda.Stream()
    gstream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(gstream):
        fwd()
    torch.cuda.current_stream().wait_stream(gstream)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        fwd()
    graph_ms, _ = time_steps(torch, graph.replay, args.steps, args.warmup)
    assert torch.equal(out.out_t, ref_t) and torch.equal(out.out_n, ref_n) and torch.equal(out.status, ref_st), \
        "graph replay differs from the eager forward"
    log(f"[bench] forward {ms_step * 1e3:.1f} us/step eager (events: median {fst['median'] * 1e3:.1f}, "
        f"stdev {fst['stdev'] * 1e3:.1f} us), {graph_ms * 1e3:.1f} us/step graph replay, "
        f"{value:.3e} neuron-events/s, status {status}")

    # ---- roofline of the forward pass: its algorithmic bytes over its
    # duration (HIP events on the launch stream, mean over the timed steps)
    alg_bytes = fwd_alg_bytes(total_ev, N, B, n_spikes)
    achieved = alg_bytes / (fst["mean"] * 1e-3) / 1e9
    traffic, traffic_per_kernel = measured_traffic()
    l2 = measured_l2()

    # ---- sequential GPU baseline (same ABI, same inputs)
    seq = lif.forward(d_t, d_s, d_n, d_W, P, sequential=True, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(seq.out_n, out.out_n), "sequential and parallel spike counts differ"
    seq_ms, _ = time_steps(torch, lambda: lif.forward(d_t, d_s, d_n, d_W, P, sequential=True, ws=ws, out=seq),
                           args.seq_steps, 0)
    log(f"[bench] sequential {seq_ms:.3f} ms/step, speedup {seq_ms / ms_step:.1f}x")

    # ---- backward pass on the same batch (dL/dt ~ N(0,1) on every spike)
    rng = np.random.default_rng(1)
    valid = np.isfinite(out.out_t.cpu().numpy())
    g = d((rng.standard_normal(valid.shape) * valid).astype(np.float32))
    bws = torch.empty(lif.lif_layer_backward_workspace_size(B, E, C, N, pc), dtype=torch.uint8, device=dev)
    bwd_ms, bev = time_steps(torch, lambda: lif.backward(d_t, d_s, d_n, d_W, out, g, P, ws=bws),
                             max(5, args.steps // 5), 3)
    log(f"[bench] backward {bwd_ms * 1e3:.1f} us/step")
    del ws, bws

    # ---- the other workloads (extra keys; the headline stays the one above)
    extras = {}
    if not args.no_extras:
        st, wu = max(3, args.steps // 10), 2
        made = {}

        def cfg(name):                                       # each config built once, when first needed
            if name not in made:
                made[name] = getattr(W, name)()
            return made[name]
        c3 = cfg("config3")
        jobs = {
            "c3_layer1": lambda: run_workload(torch, lif, d, "700->512 layer 1 of 700->512->512, B=128, ~10k events",
                                              c3.events, c3.layers[0].WT, lif.Params(s_max=128), st, wu, 1),
            "c4": lambda: run_workload(torch, lif, d, "2312->1024, B=64, ~20k events in 3 bursts",
                                       cfg("config4").events, cfg("config4").layers[0].WT, lif.Params(s_max=64), st,
                                       wu, 1),
            "c5_hidden": lambda: run_workload(torch, lif, d, "32768->2048, B=16, ~100k events (stated gain 4)",
                                              cfg("config5").events, cfg("config5").layers[0].WT,
                                              lif.Params(s_max=64), st, wu, 1, backward=True),
            # gain 16: the driven variant of the parity tests
            "c5_hidden_driven": lambda: run_workload(torch, lif, d, "32768->2048, B=16, ~100k events, gain 16",
                                                     cfg("config5").events,
                                                     (cfg("config5").layers[0].WT * 4.0).astype(np.float32),
                                                     lif.Params(s_max=64), st, wu, 1, backward=True),
            "train_step_c3": lambda: train_step(torch, lif, d, c3, st, wu),
            "train_step_c3_reg": lambda: train_step(torch, lif, d, c3, st, wu, "reg"),
            "train_step_c3_delays": lambda: train_step(torch, lif, d, c3, st, wu, "delays"),
            "train_step_c3_reg_delays": lambda: train_step(torch, lif, d, c3, st, wu, "reg_delays"),
            "chunk_mode_c2": lambda: chunk_study(torch, lif, d, ev, WT, st, wu, seq_ms),
            "delays_c2": lambda: delay_study(torch, lif, d, ev, WT, st, wu, 1),
        }
        pick = [x for x in args.extras.split(",") if x] or list(jobs)
        unknown = [x for x in pick if x not in jobs]
        if unknown:
            print(f"bench.py: unknown --extras {unknown}; known: {list(jobs)}", file=sys.stderr)
            sys.exit(2)
        for name in pick:
            extras[name] = jobs[name]()
        del c3, made, jobs

    # ---- float64 CPU oracle on the host cores (bounded samples)
    cpu = None
    cpu1 = None
    if not args.no_cpu_baseline:
        ncores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
        ncores = max(1, min(int(ncores), 16))
        rate, per, reps = cpu_oracle(ev, WT, ncores, args.cpu_seconds, B, N)
        cpu = {"value": rate, "unit": "neuron-events/s", "cores": ncores, "kind": "oracle",
               "sample": f"the full workload (32 samples x 256 neurons, {total_ev} events), repeated {reps} "
                         f"times, {per:.3f} s each; float64, one thread per core over (sample, neuron)"}
        rate1, per1, reps1 = cpu_oracle(ev, WT, 1, args.cpu_seconds / 2, 4, N)
        cpu1 = {"value": rate1, "unit": "neuron-events/s", "cores": 1, "kind": "oracle",
                "sample": f"4 samples x 256 neurons ({int(ev.ev_n[:4].sum())} events), repeated {reps1} times, "
                          f"{per1:.3f} s each; float64, one thread"}
        log(f"[bench] cpu oracle {per:.3f} s/forward on {ncores} threads; {rate1:.3e} neuron-events/s on one")

    line = {
        "metric": "neuron-events/s fwd (700->256, B=32)",
        "value": value,
        "unit": "neuron-events/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "step_event_ms": fst,
        "ms_per_step_graph_replay": graph_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "io_dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "LIF layer 700->256, B=32, 1 s lognormal-Poisson input (~5k events/sample), "
                               "tau_m 20 ms, tau_s 5 ms, threshold 1, reset 0",
                   "batch": B, "c_in": C, "n_out": N, "events": total_ev, "e_max": E,
                   "neuron_events": neuron_events, "spikes": n_spikes, "s_max": P.s_max},
        "roofline": {"bound": "hbm", "kernel": "forward pass (" + " + ".join(FORWARD_KERNELS) + ")",
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": traffic, "alg_bytes_per_launch": alg_bytes, "launch_us": fst["mean"] * 1e3,
                     "traffic_per_kernel": traffic_per_kernel, "l2_hit_rate": l2},
        "hbm_frac_forward": alg_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "kernels_us": kern_us,
        "sequential_ms": seq_ms,
        "speedup_vs_sequential": seq_ms / ms_step,
        "backward_ms": bwd_ms,
        "backward_event_ms": stats_ms(bev),
        "status": status,
        "other_workloads": extras,
        "cpu_baseline": cpu,
        "cpu_baseline_1thread": cpu1,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
