"""Benchmark of the event-driven LIF layer forward pass on one MI355X.

Workload: one LIF layer, 700 input channels -> 256 neurons, batch 32, 1 s per
sample, lognormal-rate Poisson input channels (~5k events per sample),
W ~ N(0,1) * 4/sqrt(700), tau_m = 20 ms, tau_s = 5 ms, threshold 1, hard
reset to 0 (synthetic, seeded).  A step is one forward pass of the layer
(decays, weight gather, segment scan, interval checks, root solves, resets,
outputs) over the batch, with all inputs resident in HBM.

Prints one JSON line: throughput in neuron-events/s (N_out * sum of events
per sample, per second), the roofline of the dominant kernel, the speedup
over the sequential one-thread-per-neuron GPU event loop, the backward time,
and the float64 CPU oracle timed on the host cores.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0     # MI355X HBM3E, GB/s


def log(*a):
    print(*a, file=sys.stderr, flush=True)


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_forward_700x256_b32.txt")
KERNEL_SOURCES = ("lif_forward.hip", "lif_common.hpp", "lif_host.hpp", "lif_walk.hpp")


def kernel_sources_sha256() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2603_13283_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(kernel: str):
    """HBM bytes per launch of `kernel` from the rocprofv3 FETCH_SIZE and
    WRITE_SIZE runs summarised in profiles/ (already scaled by the copy-probe
    factors), or None when they are missing or were taken on other kernel
    sources than the ones built now."""
    try:
        lines = open(TRAFFIC_FILE).read().splitlines()
    except OSError:
        return None
    sha = None
    for ln in lines:
        if ln.startswith("sources_sha256:"):
            sha = ln.split(":", 1)[1].strip()
        parts = ln.split()
        if sha and len(parts) == 3 and parts[0] == kernel:
            if sha != kernel_sources_sha256():
                return None
            return int(parts[1]) + int(parts[2])
    return None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--seq-steps", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="CPU oracle baseline: repeat the full-batch forward until this much time has passed")
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
    cfg = W.config2()
    ev, WT = cfg.events, cfg.layers[0].WT
    B, E = ev.ev_t.shape
    C, N = WT.shape
    total_ev = int(ev.ev_n.sum())
    neuron_events = N * total_ev
    P = lif.Params(s_max=64)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    d_t, d_s, d_n, d_W = t(ev.ev_t), t(ev.ev_src), t(ev.ev_n), t(WT)
    pc = P.c()
    ws = torch.empty(lif.lif_layer_forward_workspace_size(B, E, C, N, pc), dtype=torch.uint8, device=dev)
    out = lif.forward(d_t, d_s, d_n, d_W, P, ws=ws)
    torch.cuda.synchronize()
    log(f"[bench] {cfg.name}: B={B} E_max={E} events={total_ev} N={N} neuron-events={neuron_events} "
        f"lib={lif.lif_version()}")

    # ---- per-kernel durations: eager launches bracketed by HIP events on the
    # launch stream (the library's kernel timer)
    lif.lif_timer_enable(True)
    for _ in range(args.warmup):
        lif.forward(d_t, d_s, d_n, d_W, P, ws=ws, out=out)
    torch.cuda.synchronize()
    lif.lif_timer_enable(True)
    for _ in range(args.steps):
        lif.forward(d_t, d_s, d_n, d_W, P, ws=ws, out=out)
    torch.cuda.synchronize()
    kern = lif.lif_timer_read()
    lif.lif_timer_enable(False)
    log(f"[bench] kernels: " + ", ".join(f"{k}={v[0] / v[1] * 1e3:.1f}us" for k, v in kern.items()))

    # ---- eager forward steps (no timer)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        lif.forward(d_t, d_s, d_n, d_W, P, ws=ws, out=out)
    torch.cuda.synchronize()
    eager_ms = (time.perf_counter() - t0) / args.steps * 1e3
    ref_t, ref_n, ref_st = out.out_t.clone(), out.out_n.clone(), out.status.clone()

    # ---- timed steps: the forward call captured once in a HIP graph and
    # replayed (the call allocates nothing and issues only kernel launches)
    gstream = torch.cuda.Stream()
    gstream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(gstream):
        lif.forward(d_t, d_s, d_n, d_W, P, ws=ws, out=out)
    torch.cuda.current_stream().wait_stream(gstream)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        lif.forward(d_t, d_s, d_n, d_W, P, ws=ws, out=out)
    for _ in range(args.warmup):
        graph.replay()
    torch.cuda.synchronize()
    assert torch.equal(out.out_t, ref_t) and torch.equal(out.out_n, ref_n) and torch.equal(out.status, ref_st), \
        "graph replay differs from the eager forward"
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        graph.replay()
    torch.cuda.synchronize()
    graph_ms = (time.perf_counter() - t0) / args.steps * 1e3
    # The reported step is the plain (eager) library call.
    ms_step = eager_ms
    value = neuron_events / (ms_step * 1e-3)
    status = out.status.cpu().numpy().tolist()
    n_spikes = int(out.out_n.sum().item())
    log(f"[bench] forward {ms_step * 1e3:.1f} us/step eager, {graph_ms * 1e3:.1f} us/step graph replay, "
        f"{value:.3e} neuron-events/s, status {status}")

    # ---- roofline of the dominant kernel.  Algorithmic bytes per launch:
    #   aggregate, check: every event record (time + source, 8 B) and one
    #     float32 weight per neuron-event (4 B) -- both passes gather the
    #     whole W^T row slice of every event;
    #   carry: one float64 (V, I) aggregate read and one carry written per
    #     (sample, segment, neuron);
    #   records: per record its entering state (16 B), the 16 weights, event
    #     times and decay records of its sub-block (4 + 4 + 32 B each) and the
    #     record written (17 x 40 B);
    #   resolve: per walked sub-block, for each of its 16 intervals, the
    #     record's state and crossing data (16 + 24 B) and the interval's
    #     start time (4 B); plus 8 B per spike and 4 B per count.
    S = (E + 63) // 64                       # 64-event scan segments
    walked = status[4]
    alg = {"prep": B * S * 64 * 32 + total_ev * 4 + B * N * P.s_max * 8,
           "aggregate": total_ev * (8 + 4 * N),
           "check": total_ev * (8 + 4 * N),
           "carry": B * S * N * 32,
           "records": walked * (16 + 16 * 40 + 17 * 40),
           "resolve": walked * 16 * (16 + 24 + 4) + n_spikes * 8 + B * N * 4}
    kern_us = {k: v[0] / v[1] * 1e3 for k, v in kern.items()}
    dom_name = max(kern_us, key=kern_us.get)
    dom_us = kern_us[dom_name]
    alg_bytes = alg.get(dom_name, 0)
    achieved = alg_bytes / (dom_us * 1e-6) / 1e9
    fwd_alg_bytes = total_ev * (8 + 4 * N) + B * N * 4 + n_spikes * 8
    traffic = measured_traffic(dom_name)

    # ---- sequential GPU baseline (same ABI, same inputs)
    seq = lif.forward(d_t, d_s, d_n, d_W, P, sequential=True, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(seq.out_n, out.out_n), "sequential and parallel spike counts differ"
    ts0 = time.perf_counter()
    for _ in range(args.seq_steps):
        lif.forward(d_t, d_s, d_n, d_W, P, sequential=True, ws=ws, out=seq)
    torch.cuda.synchronize()
    seq_ms = (time.perf_counter() - ts0) / args.seq_steps * 1e3
    log(f"[bench] sequential {seq_ms:.3f} ms/step, speedup {seq_ms / ms_step:.1f}x")

    # ---- backward pass on the same batch (dL/dt ~ N(0,1) on every spike)
    rng = np.random.default_rng(1)
    valid = np.isfinite(out.out_t.cpu().numpy())
    g = t((rng.standard_normal(valid.shape) * valid).astype(np.float32))
    bws = torch.empty(lif.lif_layer_backward_workspace_size(B, E, C, N, pc), dtype=torch.uint8, device=dev)
    for _ in range(3):
        lif.backward(d_t, d_s, d_n, d_W, out, g, P, ws=bws)
    torch.cuda.synchronize()
    tb0 = time.perf_counter()
    nb = max(5, args.steps // 5)
    for _ in range(nb):
        lif.backward(d_t, d_s, d_n, d_W, out, g, P, ws=bws)
    torch.cuda.synchronize()
    bwd_ms = (time.perf_counter() - tb0) / nb * 1e3
    log(f"[bench] backward {bwd_ms * 1e3:.1f} us/step")

    # ---- float64 CPU oracle on the host cores (full batch, repeated)
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        ncores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
        ncores = max(1, min(int(ncores), 16))
        OP = oracle.LifParams(s_max=64)
        oracle.forward(ev.ev_t[:1], ev.ev_src[:1], ev.ev_n[:1], WT, OP, nthreads=ncores)
        reps = 0
        c0 = time.perf_counter()
        while reps < 3 or time.perf_counter() - c0 < args.cpu_seconds:
            oracle.forward(ev.ev_t, ev.ev_src, ev.ev_n, WT, OP, nthreads=ncores)
            reps += 1
        cpu_s = (time.perf_counter() - c0) / reps
        cpu = {"value": neuron_events / cpu_s, "unit": "neuron-events/s", "cores": ncores, "kind": "oracle",
               "sample": f"the full workload (32 samples x 256 neurons, {total_ev} events) repeated {reps} times, "
                         f"{cpu_s:.3f} s each, float64, one thread per core over (sample, neuron)"}
        log(f"[bench] cpu oracle {cpu_s:.3f} s/forward on {ncores} threads")

    line = {
        "metric": "neuron-events/s fwd (700->256, B=32)",
        "value": value,
        "unit": "neuron-events/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
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
        "roofline": {"bound": "hbm", "kernel": dom_name, "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "alg_bytes_per_launch": alg_bytes, "kernel_us": dom_us},
        "hbm_frac_forward": fwd_alg_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "kernels_us": kern_us,
        "sequential_ms": seq_ms,
        "speedup_vs_sequential": seq_ms / ms_step,
        "backward_ms": bwd_ms,
        "status": status,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
