"""float64 CPU oracle for the event-driven LIF layer (test infrastructure).

Only the test suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg
of ``bench.py`` may import this package.  The GPU library never links,
imports or calls it, and this package never imports the GPU library.

Two independent implementations live here:

* ``lif_oracle.c`` (compiled with gcc into ``liblif_oracle.so``): the serial
  event loop of the paper in float64, threaded over (sample, neuron) items;
  forward, backward (implicit differentiation through the resets) and the
  layer merge.  Wrapped below with ctypes + numpy.
* ``ref.py``: the same definitions in pure Python loops for tiny inputs.
* ``loss.py``: the paper's readout loss and spike-count regularisers
  (numpy, float64).

``lif_oracle.c`` also holds the chunk mode of Sec. 3.2.1 (K events per
iteration, a budget of C iterations, work counters of Appendix G) and the
layer with learnable synaptic delays (Sec. 3.1 Eq. spike_input: a queue per
neuron ordered by arrival time, App. E.2).

Functions whose results cannot be pinned independently would say
"parity unpinned" here; at present every output (spike times, counts, I at
spike, weight and input-time gradients, merged queues) has an independent pin
in ``tests/test_oracle_pins.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lif_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liblif_oracle.so")
_lib = None

TIE_BAND = 1e-6


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc (plain -O2, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread",
                               "-D_DEFAULT_SOURCE", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class _Params(ctypes.Structure):
    _fields_ = [("tau_mem", ctypes.c_double), ("tau_syn", ctypes.c_double),
                ("v_th", ctypes.c_double), ("v_reset", ctypes.c_double),
                ("t_end", ctypes.c_double), ("s_max", ctypes.c_int32),
                ("solver_reg", ctypes.c_double), ("tie_band", ctypes.c_double)]


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
            build()
        _lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        _lib.or_forward.argtypes = [P, P, P, ctypes.c_int, ctypes.c_int, P, ctypes.c_int, ctypes.c_int,
                                    ctypes.POINTER(_Params), ctypes.c_int, P, P, P, P, P, P, P]
        _lib.or_forward.restype = ctypes.c_int
        _lib.or_forward_chunked.argtypes = [P, P, P, ctypes.c_int, ctypes.c_int, P, ctypes.c_int, ctypes.c_int,
                                            ctypes.POINTER(_Params), ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                            P, P, P, P, P, P, P, P, P]
        _lib.or_forward_chunked.restype = ctypes.c_int
        _lib.or_backward.argtypes = [P, P, P, ctypes.c_int, ctypes.c_int, P, ctypes.c_int, ctypes.c_int,
                                     ctypes.POINTER(_Params), ctypes.c_int, P, P, P, P, P, P, P]
        _lib.or_backward.restype = ctypes.c_int
        _lib.or_delay_queues.argtypes = [P, P, P, ctypes.c_int, ctypes.c_int, P, ctypes.c_int, ctypes.c_int, P, P]
        _lib.or_delay_queues.restype = ctypes.c_int
        _lib.or_forward_delayed.argtypes = [P, P, P, ctypes.c_int, ctypes.c_int, P, P, ctypes.c_int, ctypes.c_int,
                                            ctypes.POINTER(_Params), ctypes.c_int, P, P, P, P, P, P, P]
        _lib.or_forward_delayed.restype = ctypes.c_int
        _lib.or_backward_delayed.argtypes = [P, P, P, ctypes.c_int, ctypes.c_int, P, P, ctypes.c_int, ctypes.c_int,
                                             ctypes.POINTER(_Params), ctypes.c_int, P, P, P, P, P, P, P, P]
        _lib.or_backward_delayed.restype = ctypes.c_int
        _lib.or_trace.argtypes = [P, P, ctypes.c_int, P, ctypes.c_int, ctypes.c_int,
                                  ctypes.POINTER(_Params), P, P]
        _lib.or_trace.restype = ctypes.c_int
        _lib.or_merge.argtypes = [P, P, ctypes.c_int, ctypes.c_int, ctypes.c_int, P, P, P, P, ctypes.c_int]
        _lib.or_merge.restype = ctypes.c_int
        D = ctypes.c_double
        _lib.or_check_interval.argtypes = [ctypes.POINTER(_Params), D, D, D, ctypes.POINTER(D), ctypes.POINTER(D)]
        _lib.or_check_interval.restype = ctypes.c_int
        _lib.or_solve_root.argtypes = [ctypes.POINTER(_Params), D, D, D]
        _lib.or_solve_root.restype = D
    return _lib


@dataclass
class LifParams:
    tau_mem: float = 0.02
    tau_syn: float = 0.005
    v_th: float = 1.0
    v_reset: float = 0.0
    t_end: float = float("inf")
    s_max: int = 64
    solver_reg: float = 0.01
    tie_band: float = TIE_BAND

    def c(self) -> _Params:
        return _Params(self.tau_mem, self.tau_syn, self.v_th, self.v_reset, self.t_end,
                       int(self.s_max), self.solver_reg, self.tie_band)


@dataclass
class ForwardResult:
    out_t: np.ndarray    # float64 [B, N, s_max], +inf padding
    out_i: np.ndarray    # float64 [B, N, s_max], I at each spike
    out_n: np.ndarray    # int32 [B, N]
    capped: np.ndarray   # int32 [B, N]
    tie_t: np.ndarray    # float64 [B, N]: start of first near-tie interval, +inf if none
    min_gap: np.ndarray  # float64 [B, N]: smallest |V_max - V_th| over checked intervals
    out_k: np.ndarray    # int32 [B, N, s_max]: input events consumed before each spike, 0 padding

    def rounded(self) -> "ForwardResult":
        """The same result with spike times and currents rounded to float32
        (what a float32 forward hands to a backward pass), widened again."""
        return ForwardResult(self.out_t.astype(np.float32).astype(np.float64),
                             self.out_i.astype(np.float32).astype(np.float64), self.out_n, self.capped,
                             self.tie_t, self.min_gap, self.out_k)

    def select(self, keep) -> "ForwardResult":
        """The samples selected by a boolean mask over the batch."""
        return ForwardResult(self.out_t[keep], self.out_i[keep], self.out_n[keep], self.capped[keep],
                             self.tie_t[keep], self.min_gap[keep], self.out_k[keep])


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _nthreads(n: Optional[int]) -> int:
    if n is None:
        n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    return max(1, int(n))


def forward(ev_t, ev_src, ev_n, WT, params: LifParams = LifParams(), nthreads: Optional[int] = None) -> ForwardResult:
    """Serial float64 forward pass of one LIF layer over a padded batch."""
    lib = _load()
    ev_t = np.ascontiguousarray(ev_t, dtype=np.float32)
    ev_src = np.ascontiguousarray(ev_src, dtype=np.int32)
    ev_n = np.ascontiguousarray(ev_n, dtype=np.int32)
    WT = np.ascontiguousarray(WT, dtype=np.float32)
    B, E = ev_t.shape
    C, N = WT.shape
    S = int(params.s_max)
    out_t = np.empty((B, N, S), np.float64)
    out_i = np.empty((B, N, S), np.float64)
    out_k = np.empty((B, N, S), np.int32)
    out_n = np.empty((B, N), np.int32)
    capped = np.empty((B, N), np.int32)
    tie_t = np.empty((B, N), np.float64)
    min_gap = np.empty((B, N), np.float64)
    p = params.c()
    rc = lib.or_forward(_ptr(ev_t), _ptr(ev_src), _ptr(ev_n), B, E, _ptr(WT), C, N, ctypes.byref(p),
                        _nthreads(nthreads), _ptr(out_t), _ptr(out_i), _ptr(out_k), _ptr(out_n), _ptr(capped),
                        _ptr(tie_t), _ptr(min_gap))
    if rc != 0:
        raise ValueError(f"oracle forward rejected its arguments (rc={rc})")
    return ForwardResult(out_t, out_i, out_n, capped, tie_t, min_gap, out_k)


def forward_chunked(ev_t, ev_src, ev_n, WT, K: int, C: int, params: LifParams = LifParams(),
                    nthreads: Optional[int] = None):
    """Chunk-mode forward (K events per chunk iteration, at most C
    iterations per neuron; Sec. 3.2.1 speculative execution and fixed
    budget).  Returns (ForwardResult, consumed [B, N], processed [B, N])."""
    lib = _load()
    ev_t = np.ascontiguousarray(ev_t, dtype=np.float32)
    ev_src = np.ascontiguousarray(ev_src, dtype=np.int32)
    ev_n = np.ascontiguousarray(ev_n, dtype=np.int32)
    WT = np.ascontiguousarray(WT, dtype=np.float32)
    B, E = ev_t.shape
    C_in, N = WT.shape
    S = int(params.s_max)
    out_t = np.empty((B, N, S), np.float64)
    out_i = np.empty((B, N, S), np.float64)
    out_k = np.empty((B, N, S), np.int32)
    out_n = np.empty((B, N), np.int32)
    capped = np.empty((B, N), np.int32)
    tie_t = np.empty((B, N), np.float64)
    min_gap = np.empty((B, N), np.float64)
    consumed = np.empty((B, N), np.int32)
    processed = np.empty((B, N), np.int32)
    p = params.c()
    rc = lib.or_forward_chunked(_ptr(ev_t), _ptr(ev_src), _ptr(ev_n), B, E, _ptr(WT), C_in, N, ctypes.byref(p),
                                int(K), int(C), _nthreads(nthreads), _ptr(out_t), _ptr(out_i), _ptr(out_k),
                                _ptr(out_n), _ptr(capped), _ptr(tie_t), _ptr(min_gap), _ptr(consumed),
                                _ptr(processed))
    if rc != 0:
        raise ValueError(f"oracle chunked forward rejected its arguments (rc={rc})")
    return ForwardResult(out_t, out_i, out_n, capped, tie_t, min_gap, out_k), consumed, processed


def backward(ev_t, ev_src, ev_n, WT, fwd: ForwardResult, grad_out_t, params: LifParams = LifParams(),
             nthreads: Optional[int] = None):
    """float64 gradients (grad_WT [C_in, N], grad_ev_t [B, E_max]) of
    L = sum grad_out_t * out_t, through a forward result for the same inputs
    (spike times, currents at the spikes and the consumed-event counts)."""
    lib = _load()
    ev_t = np.ascontiguousarray(ev_t, dtype=np.float32)
    ev_src = np.ascontiguousarray(ev_src, dtype=np.int32)
    ev_n = np.ascontiguousarray(ev_n, dtype=np.int32)
    WT = np.ascontiguousarray(WT, dtype=np.float32)
    B, E = ev_t.shape
    C, N = WT.shape
    g = np.ascontiguousarray(grad_out_t, dtype=np.float64)
    gW = np.empty((C, N), np.float64)
    gT = np.empty((B, E), np.float64)
    p = params.c()
    rc = lib.or_backward(_ptr(ev_t), _ptr(ev_src), _ptr(ev_n), B, E, _ptr(WT), C, N, ctypes.byref(p),
                         _nthreads(nthreads), _ptr(np.ascontiguousarray(fwd.out_t, dtype=np.float64)),
                         _ptr(np.ascontiguousarray(fwd.out_i, dtype=np.float64)),
                         _ptr(np.ascontiguousarray(fwd.out_k, dtype=np.int32)),
                         _ptr(np.ascontiguousarray(fwd.out_n, dtype=np.int32)),
                         _ptr(g), _ptr(gW), _ptr(gT))
    if rc != 0:
        raise RuntimeError(f"oracle backward failed (rc={rc})")
    return gW, gT


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def delay_queues(ev_t, ev_src, ev_n, DT):
    """Each neuron's queue of arrivals (Sec. 3.1 Eq. spike_input, App. E.2):
    event k of sample b reaches neuron i at fl32(t_k + DT[src_k, i]), ordered
    by (arrival, k).  Returns q_t float32 [B, N, E_max] and q_k int32 (the
    sample's event index); entries past ev_n[b] are 0."""
    ev_t, ev_src, ev_n, DT = _f32(ev_t), _i32(ev_src), _i32(ev_n), _f32(DT)
    B, E = ev_t.shape
    C, N = DT.shape
    q_t = np.zeros((B, N, E), np.float32)
    q_k = np.zeros((B, N, E), np.int32)
    rc = _load().or_delay_queues(_ptr(ev_t), _ptr(ev_src), _ptr(ev_n), B, E, _ptr(DT), C, N, _ptr(q_t), _ptr(q_k))
    if rc != 0:
        raise RuntimeError(f"oracle delay queues failed (rc={rc})")
    return q_t, q_k


def forward_delayed(ev_t, ev_src, ev_n, WT, DT, params: LifParams = LifParams(),
                    nthreads: Optional[int] = None) -> ForwardResult:
    """Serial float64 forward of a layer with synaptic delays DT [C_in, N]:
    every neuron runs the serial simulation on its own arrival queue (out_k
    counts events of that queue)."""
    lib = _load()
    ev_t, ev_src, ev_n, WT, DT = _f32(ev_t), _i32(ev_src), _i32(ev_n), _f32(WT), _f32(DT)
    B, E = ev_t.shape
    C, N = WT.shape
    assert DT.shape == WT.shape
    S = int(params.s_max)
    out_t = np.empty((B, N, S), np.float64)
    out_i = np.empty((B, N, S), np.float64)
    out_k = np.empty((B, N, S), np.int32)
    out_n = np.empty((B, N), np.int32)
    capped = np.empty((B, N), np.int32)
    tie_t = np.empty((B, N), np.float64)
    min_gap = np.empty((B, N), np.float64)
    p = params.c()
    rc = lib.or_forward_delayed(_ptr(ev_t), _ptr(ev_src), _ptr(ev_n), B, E, _ptr(WT), _ptr(DT), C, N,
                                ctypes.byref(p), _nthreads(nthreads), _ptr(out_t), _ptr(out_i), _ptr(out_k),
                                _ptr(out_n), _ptr(capped), _ptr(tie_t), _ptr(min_gap))
    if rc != 0:
        raise ValueError(f"oracle delayed forward rejected its arguments (rc={rc})")
    return ForwardResult(out_t, out_i, out_n, capped, tie_t, min_gap, out_k)


def backward_delayed(ev_t, ev_src, ev_n, WT, DT, fwd: ForwardResult, grad_out_t,
                     params: LifParams = LifParams(), nthreads: Optional[int] = None):
    """float64 gradients (grad_WT, grad_DT [C_in, N], grad_ev_t [B, E_max])
    of L = sum grad_out_t * out_t for a layer with delays, through a delayed
    forward result for the same inputs."""
    lib = _load()
    ev_t, ev_src, ev_n, WT, DT = _f32(ev_t), _i32(ev_src), _i32(ev_n), _f32(WT), _f32(DT)
    B, E = ev_t.shape
    C, N = WT.shape
    g = np.ascontiguousarray(grad_out_t, dtype=np.float64)
    gW = np.empty((C, N), np.float64)
    gD = np.empty((C, N), np.float64)
    gT = np.empty((B, E), np.float64)
    p = params.c()
    rc = lib.or_backward_delayed(_ptr(ev_t), _ptr(ev_src), _ptr(ev_n), B, E, _ptr(WT), _ptr(DT), C, N,
                                 ctypes.byref(p), _nthreads(nthreads),
                                 _ptr(np.ascontiguousarray(fwd.out_t, dtype=np.float64)),
                                 _ptr(np.ascontiguousarray(fwd.out_i, dtype=np.float64)),
                                 _ptr(np.ascontiguousarray(fwd.out_k, dtype=np.int32)),
                                 _ptr(np.ascontiguousarray(fwd.out_n, dtype=np.int32)),
                                 _ptr(g), _ptr(gW), _ptr(gD), _ptr(gT))
    if rc != 0:
        raise RuntimeError(f"oracle delayed backward failed (rc={rc})")
    return gW, gD, gT


def trace(ev_t_row, ev_src_row, n, WT, i, params: LifParams = LifParams()):
    """(V, I) just after each of the first n events for neuron i of one sample."""
    lib = _load()
    ev_t_row = np.ascontiguousarray(ev_t_row, dtype=np.float32)
    ev_src_row = np.ascontiguousarray(ev_src_row, dtype=np.int32)
    WT = np.ascontiguousarray(WT, dtype=np.float32)
    V = np.zeros(max(n, 1), np.float64)
    I = np.zeros(max(n, 1), np.float64)
    p = params.c()
    ns = lib.or_trace(_ptr(ev_t_row), _ptr(ev_src_row), int(n), _ptr(WT), WT.shape[1], int(i),
                      ctypes.byref(p), _ptr(V), _ptr(I))
    return V[:n], I[:n], int(ns)


def check_interval(V0: float, I0: float, length: float, params: LifParams = LifParams()):
    """Interval rule of Sec. 3.2.2 from state (V0, I0): (crossing, bracket_hi, V_max)."""
    lib = _load()
    hi = ctypes.c_double()
    vmax = ctypes.c_double()
    p = params.c()
    c = lib.or_check_interval(ctypes.byref(p), float(V0), float(I0), float(length), ctypes.byref(hi),
                              ctypes.byref(vmax))
    return bool(c), hi.value, vmax.value


def solve_root(V0: float, I0: float, hi: float, params: LifParams = LifParams()) -> float:
    """Smallest float64 offset tau in (0, hi] with V(tau) >= V_th."""
    p = params.c()
    return float(_load().or_solve_root(ctypes.byref(p), float(V0), float(I0), float(hi)))


def merge(out_t32, out_n, E2_max: int):
    """Per-sample merge of spike lists (float32 times) into sorted queues.
    Returns (ev_t2, ev_src2, ev_n2, perm, overflow)."""
    lib = _load()
    out_t32 = np.ascontiguousarray(out_t32, dtype=np.float32)
    out_n = np.ascontiguousarray(out_n, dtype=np.int32)
    B, N, S = out_t32.shape
    ev_t2 = np.empty((B, E2_max), np.float32)
    ev_src2 = np.empty((B, E2_max), np.int32)
    ev_n2 = np.empty(B, np.int32)
    perm = np.empty((B, E2_max), np.int32)
    rc = lib.or_merge(_ptr(out_t32), _ptr(out_n), B, N, S, _ptr(ev_t2), _ptr(ev_src2), _ptr(ev_n2),
                      _ptr(perm), int(E2_max))
    return ev_t2, ev_src2, ev_n2, perm, bool(rc)


def first_spike_ce(out_t_first, spiked, labels, tau0: float, t_silent: float):
    """Readout loss: logits_c = -t_c / tau0 with t_c the first spike time of
    readout neuron c (t_silent if it never fires); mean softmax
    cross-entropy over the batch.  Returns (loss, dL/dt_first) in float64;
    silent neurons get a zero gradient (their time is a constant)."""
    t = np.where(spiked, np.asarray(out_t_first, np.float64), t_silent)
    z = -t / tau0
    z = z - z.max(axis=1, keepdims=True)
    pz = np.exp(z)
    pz /= pz.sum(axis=1, keepdims=True)
    B = t.shape[0]
    loss = -np.mean(np.log(pz[np.arange(B), labels]))
    onehot = np.zeros_like(pz)
    onehot[np.arange(B), labels] = 1.0
    g = (pz - onehot) / B * (-1.0 / tau0)
    g = np.where(spiked, g, 0.0)
    return float(loss), g
