"""Seeded synthetic input generators for the event-driven LIF layer.

This module only draws random numbers and lays them out: it holds none of the
method's arithmetic (no decays, no membrane dynamics, no spike solving).  Both
the float64 CPU oracle and the GPU path consume exactly the arrays produced
here, so every parity comparison starts from bit-identical float32 inputs.

Event streams stand in for the paper's audio/event-camera datasets (SHD/SSC,
700 channels, at most 14000 input spikes per sample; Appendix E.4), which are
not available here.  Every stream is a per-sample queue of (time, source)
pairs sorted by (float32 time, source), padded with +inf times and source 0
(Appendix E.2: sorted per-sample event queues).

Randomness: numpy ``Generator(PCG64)`` children of ``SeedSequence(seed)``,
spawned in the fixed order [weights, events, labels, spare].
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

# Constants shared by every workload (the paper's hyperparameter table in App. E,
# "System hyperparameters across the 3 datasets used": tau_m = 20 ms,
# tau_s = 5 ms, threshold 1, reset 0, solver regularisation 0.01).
TAU_MEM = 0.02
TAU_SYN = 0.005
V_TH = 1.0
V_RESET = 0.0
SOLVER_REG = 0.01


@dataclass
class EventBatch:
    """Padded per-sample event queues.

    ev_t  : float32 [B, E_max], sorted per row, +inf padding
    ev_src: int32   [B, E_max], source channel per event, 0 padding
    ev_n  : int32   [B], number of real events per sample
    """

    ev_t: np.ndarray
    ev_src: np.ndarray
    ev_n: np.ndarray

    @property
    def B(self) -> int:
        return int(self.ev_t.shape[0])

    @property
    def E_max(self) -> int:
        return int(self.ev_t.shape[1])

    @property
    def total_events(self) -> int:
        return int(self.ev_n.sum())


@dataclass
class Layer:
    """One fully connected LIF layer: weights in W^T layout [C_in, N_out]."""

    WT: np.ndarray  # float32 [C_in, N_out]; WT[c, i] = w_{i c}

    @property
    def C_in(self) -> int:
        return int(self.WT.shape[0])

    @property
    def N(self) -> int:
        return int(self.WT.shape[1])


@dataclass
class Workload:
    name: str
    events: EventBatch
    layers: List[Layer]
    labels: Optional[np.ndarray] = None
    T: float = 1.0
    params: dict = field(default_factory=dict)


def _rngs(seed: int):
    ss = np.random.SeedSequence(seed)
    return [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(4)]


def pack_events(times: List[np.ndarray], srcs: List[np.ndarray], e_max: Optional[int] = None) -> EventBatch:
    """Round times to float32, sort each sample by (time, src) and pad."""
    B = len(times)
    ns = [int(t.size) for t in times]
    E = max([1] + ns) if e_max is None else int(e_max)
    if any(n > E for n in ns):
        raise ValueError("e_max smaller than a sample's event count")
    ev_t = np.full((B, E), np.inf, dtype=np.float32)
    ev_src = np.zeros((B, E), dtype=np.int32)
    for b in range(B):
        t32 = np.asarray(times[b], dtype=np.float64).astype(np.float32)
        s = np.asarray(srcs[b], dtype=np.int64).astype(np.int32)
        order = np.lexsort((s, t32))
        ev_t[b, : t32.size] = t32[order]
        ev_src[b, : t32.size] = s[order]
    return EventBatch(ev_t, ev_src, np.asarray(ns, dtype=np.int32))


def gaussian_weights(rng, C_in: int, N: int, gain: float) -> np.ndarray:
    """W ~ N(0,1) * gain / sqrt(fan_in), drawn in float64, stored float32 as W^T."""
    w = rng.standard_normal((C_in, N)) * (gain / np.sqrt(C_in))
    return w.astype(np.float32)


def lognormal_poisson(rng, B: int, C: int, T: float, median_hz: float, sigma: float = 1.0):
    """Per (sample, channel) rate r = m * exp(sigma z); count ~ Poisson(r T);
    times ~ U[0, T)."""
    times, srcs = [], []
    for _ in range(B):
        r = median_hz * np.exp(sigma * rng.standard_normal(C))
        n = rng.poisson(r * T)
        src = np.repeat(np.arange(C, dtype=np.int64), n)
        t = rng.random(src.size) * T
        times.append(t)
        srcs.append(src)
    return times, srcs


def uniform_events(rng, B: int, C: int, n_events: int, T: float):
    times, srcs = [], []
    for _ in range(B):
        times.append(rng.random(n_events) * T)
        srcs.append(rng.integers(0, C, size=n_events))
    return times, srcs


def burst_events(rng, B: int, C: int = 2312, n_bursts: int = 3, window: float = 0.1,
                 active_frac: float = 0.3, mean_count: float = 9.606, sigma_t: float = 0.015):
    """Event-camera-shaped input: bursts in consecutive windows; per burst a
    fraction of channels is active, each emitting Poisson(mean_count) events
    with Gaussian times around the window centre, resampled into the window."""
    times, srcs = [], []
    n_active = int(round(active_frac * C))
    for _ in range(B):
        ts, ss = [], []
        for k in range(n_bursts):
            lo, hi = k * window, (k + 1) * window
            mu = lo + 0.5 * window
            act = rng.choice(C, size=n_active, replace=False)
            cnt = rng.poisson(mean_count, size=n_active)
            src = np.repeat(act.astype(np.int64), cnt)
            t = rng.normal(mu, sigma_t, size=src.size)
            bad = (t < lo) | (t >= hi)
            while bad.any():
                t[bad] = rng.normal(mu, sigma_t, size=int(bad.sum()))
                bad = (t < lo) | (t >= hi)
            ts.append(t)
            ss.append(src)
        times.append(np.concatenate(ts))
        srcs.append(np.concatenate(ss))
    return times, srcs


def camera_channel(p: int, y: int, x: int, H: int = 34, W: int = 34) -> int:
    """Channel id of polarity p at pixel (y, x)."""
    return p * H * W + y * W + x


# --------------------------------------------------------------------------
# The five workloads (plus scaled-down variants used by the parity tests).
# --------------------------------------------------------------------------

def config1(seed: int = 0, gain: float = 3.0) -> Workload:
    """Batch 1, 64 -> 32, exactly 256 events uniform on [0, 1) s."""
    rw, re, _, _ = _rngs(seed)
    WT = gaussian_weights(rw, 64, 32, gain)
    t, s = uniform_events(re, 1, 64, 256, 1.0)
    return Workload("c1_64x32_b1_256ev", pack_events(t, s), [Layer(WT)], T=1.0)


def config2(seed: int = 0, B: int = 32, C: int = 700, N: int = 256, median_hz: float = 4.33,
            gain: float = 4.0, T: float = 1.0) -> Workload:
    """700 -> 256, batch 32, lognormal Poisson channels (~5k events/sample)."""
    rw, re, _, _ = _rngs(seed)
    WT = gaussian_weights(rw, C, N, gain)
    t, s = lognormal_poisson(re, B, C, T, median_hz)
    return Workload(f"c2_{C}x{N}_b{B}", pack_events(t, s), [Layer(WT)], T=T)


def config3(seed: int = 0, B: int = 128, C: int = 700, H: int = 512, median_hz: float = 8.66,
            gain: float = 4.0, T: float = 1.0) -> Workload:
    """700 -> 512 -> 512, batch 128 (~10k input events/sample)."""
    rw, re, _, _ = _rngs(seed)
    W1 = gaussian_weights(rw, C, H, gain)
    W2 = gaussian_weights(rw, H, H, gain)
    t, s = lognormal_poisson(re, B, C, T, median_hz)
    return Workload(f"c3_{C}x{H}x{H}_b{B}", pack_events(t, s), [Layer(W1), Layer(W2)], T=T)


def config4(seed: int = 0, B: int = 64, N: int = 1024, gain: float = 3.0) -> Workload:
    """2x34x34 = 2312 polarity channels -> 1024, batch 64, three 100 ms bursts."""
    rw, re, _, _ = _rngs(seed)
    C = 2 * 34 * 34
    WT = gaussian_weights(rw, C, N, gain)
    t, s = burst_events(re, B, C)
    return Workload(f"c4_{C}x{N}_b{B}", pack_events(t, s), [Layer(WT)], T=0.3)


def config5(seed: int = 0, B: int = 16, C: int = 32768, H: int = 2048, n_cls: int = 20,
            median_hz: float = 1.851, g1: float = 4.0, g2: float = 4.0, T: float = 1.0) -> Workload:
    """2x128x128 = 32768 -> 2048 -> 20 readout, batch 16 (~100k events/sample)."""
    rw, re, rl, _ = _rngs(seed)
    W1 = gaussian_weights(rw, C, H, g1)
    W2 = gaussian_weights(rw, H, n_cls, g2)
    t, s = lognormal_poisson(re, B, C, T, median_hz)
    labels = rl.integers(0, n_cls, size=B).astype(np.int64)
    return Workload(f"c5_{C}x{H}x{n_cls}_b{B}", pack_events(t, s), [Layer(W1), Layer(W2)],
                    labels=labels, T=T)


def driven_single_event(weights: np.ndarray, t0: float = 0.0) -> tuple:
    """One input event at t0 onto N neurons whose single weight is weights[i]:
    B = 1, C_in = 1.  Used for the closed-form spike-time pins."""
    w = np.asarray(weights, dtype=np.float32).reshape(1, -1)
    ev = pack_events([np.array([t0])], [np.array([0])])
    return ev, w


def random_small(seed: int, B: int, C: int, N: int, n_events: int, T: float, gain: float,
                 ragged: bool = True) -> Workload:
    """Small driven case for parity tests: uniform times, optional ragged
    per-sample event counts (including empty samples)."""
    rw, re, _, _ = _rngs(seed)
    WT = gaussian_weights(rw, C, N, gain)
    times, srcs = [], []
    for b in range(B):
        n = n_events
        if ragged:
            n = int(re.integers(0, n_events + 1)) if b % 3 else n_events
        times.append(re.random(n) * T)
        srcs.append(re.integers(0, C, size=n))
    return Workload(f"small_s{seed}", pack_events(times, srcs), [Layer(WT)], T=T)


def uniform_delays(seed: int, C_in: int, N: int, d_max: float = 0.1) -> np.ndarray:
    """Synaptic delays d_ij ~ U[0, d_max) s as float32 [C_in, N] (the W^T
    layout), the initialisation of App. E.5 (delay initialisation multiplier
    0.1 s).  Drawn from the spare stream of the seed."""
    rs = _rngs(seed)[3]
    return (rs.random((C_in, N)) * d_max).astype(np.float32)
