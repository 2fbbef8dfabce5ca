"""Python binding of liblif.so, the MI355X (gfx950) event-driven LIF layer.

Argument marshalling only: every step of the forward and backward passes runs
in the library's HIP kernels.  PyTorch supplies device memory and the current
HIP stream.  The entry points carry the C names of ``include/lif.h``
(``lif_layer_forward``, ``lif_layer_forward_sequential``,
``lif_layer_backward``, ``lif_merge_spikes``, ``lif_first_spike_ce``, the
workspace-size queries, ``lif_version``); ``forward``/``backward``/``merge``
are conveniences that allocate outputs and workspace as torch tensors and
call them.

Importing this module does not touch the GPU.  Loading the library fails
loudly (``LibraryMissing``) if ``liblif.so`` has not been built: there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liblif.so")

LIF_OK = 0
LIF_ERR_ARG = -1
LIF_ERR_TAU = -2
LIF_ERR_THRESHOLD = -3
LIF_ERR_WORKSPACE = -4
LIF_ERR_HIP = -5
LIF_ERR_SIZE = -6
ERR_NAMES = {LIF_ERR_ARG: "LIF_ERR_ARG", LIF_ERR_TAU: "LIF_ERR_TAU", LIF_ERR_THRESHOLD: "LIF_ERR_THRESHOLD",
             LIF_ERR_WORKSPACE: "LIF_ERR_WORKSPACE", LIF_ERR_HIP: "LIF_ERR_HIP", LIF_ERR_SIZE: "LIF_ERR_SIZE"}

LIF_VALIDATE = 1
LIF_ROOT_GENERAL = 2
LIF_STATUS_WORDS = 8
ST_FLAGS, ST_CAPPED, ST_SPIKES, ST_CAND_BLOCKS, ST_WALKED_BLOCKS, ST_ROOT_SOLVES, ST_EVENTS, ST_POOL_FALLBACK = range(8)
WARN_SPIKE_CAP, WARN_UNSORTED, WARN_BAD_SOURCE, WARN_NONFINITE, WARN_MERGE_FULL, WARN_BAD_COUNT = 1, 2, 4, 8, 16, 32
WARN_INTERNAL = 64
WARN_BAD_DELAY = 128
LIF_MERGE_MAX = 16384

EXPORTED = ["lif_version", "lif_layer_forward_workspace_size", "lif_layer_forward",
            "lif_layer_forward_sequential", "lif_layer_forward_noalloc", "lif_layer_forward_noalloc_max_bytes",
            "lif_layer_forward_chunked",
            "lif_layer_backward_workspace_size", "lif_layer_backward",
            "lif_merge_workspace_size", "lif_merge_spikes", "lif_first_spike_ce", "lif_merge_grad",
            "lif_li_readout_workspace_size", "lif_li_readout", "lif_adam_step", "lif_spike_count_reg_workspace_size",
            "lif_spike_count_reg", "lif_spike_count_reg_backward_workspace_size", "lif_spike_count_reg_backward",
            "lif_delay_queues_workspace_size", "lif_delay_queues",
            "lif_layer_forward_delayed", "lif_layer_forward_delayed_sequential",
            "lif_layer_backward_delayed_workspace_size", "lif_layer_backward_delayed",
            "lif_spike_count_reg_delayed_workspace_size", "lif_spike_count_reg_delayed",
            "lif_spike_count_reg_delayed_backward",
            "lif_add", "lif_softplus", "lif_softplus_grad", "lif_timer_enable", "lif_timer_read"]
LIF_LI_MAX_CLASSES = 64


class LibraryMissing(RuntimeError):
    pass


class LifError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__(f"{fn} returned {ERR_NAMES.get(code, code)}")
        self.code = code


class lif_params(ctypes.Structure):
    _fields_ = [("tau_mem", ctypes.c_double), ("tau_syn", ctypes.c_double), ("v_th", ctypes.c_double),
                ("v_reset", ctypes.c_double), ("t_end", ctypes.c_double), ("s_max", ctypes.c_int32),
                ("flags", ctypes.c_uint32), ("solver_reg", ctypes.c_double), ("pool_cap", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


@dataclass
class Params:
    """Layer constants (defaults: the paper's hyperparameter table in App. E,
    SHD/SSC columns) and the per-call options of lif_params."""
    tau_mem: float = 0.02
    tau_syn: float = 0.005
    v_th: float = 1.0
    v_reset: float = 0.0
    t_end: float = math.inf
    s_max: int = 64
    solver_reg: float = 0.01
    validate: bool = False
    root_general: bool = False
    pool_cap: int = -1

    def c(self) -> lif_params:
        flags = (LIF_VALIDATE if self.validate else 0) | (LIF_ROOT_GENERAL if self.root_general else 0)
        return lif_params(self.tau_mem, self.tau_syn, self.v_th, self.v_reset, self.t_end, int(self.s_max),
                          flags, self.solver_reg, int(self.pool_cap), 0)


class lif_li_params(ctypes.Structure):
    _fields_ = [("tau_mem", ctypes.c_double), ("tau_syn", ctypes.c_double), ("tau_li", ctypes.c_double),
                ("tau_max", ctypes.c_double), ("beta", ctypes.c_double)]


@dataclass
class LiParams:
    """Readout constants: LI time constants, the weighting constant tau_li
    (inf: unweighted), the integration window tau_max and the logit
    temperature multiplier beta."""
    tau_mem: float = 0.02
    tau_syn: float = 0.005
    tau_li: float = 0.5
    tau_max: float = 1.0
    beta: float = 0.05

    def c(self) -> lif_li_params:
        return lif_li_params(self.tau_mem, self.tau_syn, self.tau_li, self.tau_max, self.beta)


class lif_adam_params(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_double), ("beta1", ctypes.c_double), ("beta2", ctypes.c_double),
                ("eps", ctypes.c_double)]


_lib = None
_P = ctypes.c_void_p
_I = ctypes.c_int
_SZ = ctypes.c_size_t
_PP = ctypes.POINTER(lif_params)


def load(path: Optional[str] = None):
    """Load liblif.so (raises LibraryMissing if it was not built)."""
    global _lib
    if _lib is not None:
        return _lib
    path = path or LIB_PATH
    if not os.path.exists(path):
        raise LibraryMissing(f"{path} not found: build it with `python -c 'import __graft_entry__ as g; g.build()'`")
    lib = ctypes.CDLL(path)
    lib.lif_version.restype = ctypes.c_char_p
    lib.lif_version.argtypes = []
    for name in ("lif_layer_forward_workspace_size", "lif_layer_backward_workspace_size"):
        f = getattr(lib, name)
        f.restype = _SZ
        f.argtypes = [_I, _I, _I, _I, _PP]
    fwd_args = [_P, _P, _P, _I, _I, _P, _I, _I, _PP, _P, _P, _P, _P, _P, _P, _SZ, _P]
    for name in ("lif_layer_forward", "lif_layer_forward_sequential"):
        f = getattr(lib, name)
        f.restype = _I
        f.argtypes = fwd_args
    lib.lif_layer_forward_chunked.restype = _I
    lib.lif_layer_forward_chunked.argtypes = [_P, _P, _P, _I, _I, _P, _I, _I, _PP, _I, _I, _P, _P, _P, _P, _P, _P, _P,
                                              _P]
    lib.lif_layer_forward_noalloc.restype = _I
    lib.lif_layer_forward_noalloc.argtypes = fwd_args[:14] + [_P]
    lib.lif_layer_forward_noalloc_max_bytes.restype = _SZ
    lib.lif_layer_forward_noalloc_max_bytes.argtypes = []
    lib.lif_layer_backward.restype = _I
    lib.lif_layer_backward.argtypes = [_P, _P, _P, _I, _I, _P, _I, _I, _PP, _P, _P, _P, _P, _P, _P, _P, _P, _SZ,
                                       _P]
    lib.lif_merge_workspace_size.restype = _SZ
    lib.lif_merge_workspace_size.argtypes = [_I, _I, _I, _I]
    lib.lif_merge_spikes.restype = _I
    lib.lif_merge_spikes.argtypes = [_P, _P, _I, _I, _I, _P, _P, _P, _P, _I, _P, _P, _SZ, _P]
    lib.lif_first_spike_ce.restype = _I
    lib.lif_first_spike_ce.argtypes = [_P, _P, _I, _I, _I, _P, ctypes.c_double, ctypes.c_double, _P, _P, _P]
    lib.lif_merge_grad.restype = _I
    lib.lif_merge_grad.argtypes = [_P, _P, _P, _I, _I, _I, _I, _P, _P]
    lib.lif_li_readout_workspace_size.restype = _SZ
    lib.lif_li_readout_workspace_size.argtypes = [_I, _I, _I, _I]
    lib.lif_li_readout.restype = _I
    lib.lif_li_readout.argtypes = [_P, _P, _P, _I, _I, _P, _I, _I, ctypes.POINTER(lif_li_params), _P, _P, _P, _P,
                                   _P, _P, _SZ, _P]
    lib.lif_spike_count_reg_workspace_size.restype = _SZ
    lib.lif_spike_count_reg_workspace_size.argtypes = [_I, _I, _I, _I]
    lib.lif_spike_count_reg.restype = _I
    lib.lif_spike_count_reg.argtypes = [_P, _P, _P, _I, _I, _P, _I, _I, _PP, _P, _P, _P, ctypes.c_double, _P, _P,
                                        _P, _P, _SZ, _P]
    lib.lif_adam_step.restype = _I
    lib.lif_adam_step.argtypes = [_P, _P, _P, _P, _SZ, ctypes.POINTER(lif_adam_params), _I, _P]
    lib.lif_spike_count_reg_backward_workspace_size.restype = _SZ
    lib.lif_spike_count_reg_backward_workspace_size.argtypes = [_I, _I, _I, _I]
    lib.lif_spike_count_reg_backward.restype = _I
    lib.lif_spike_count_reg_backward.argtypes = [_P, _P, _P, _I, _I, _P, _I, _I, _PP, _P, _P, _P, ctypes.c_double,
                                                 ctypes.c_double, ctypes.c_double, _P, _P, _P, _P, _P, _SZ, _P]
    lib.lif_spike_count_reg_delayed_workspace_size.restype = _SZ
    lib.lif_spike_count_reg_delayed_workspace_size.argtypes = [_I, _I, _I, _I]
    lib.lif_spike_count_reg_delayed.restype = _I
    lib.lif_spike_count_reg_delayed.argtypes = [_P, _P, _P, _P, _I, _I, _P, _I, _I, _PP, _P, _P, _P, ctypes.c_double,
                                                _P, _P, _P, _P, _SZ, _P]
    lib.lif_spike_count_reg_delayed_backward.restype = _I
    lib.lif_spike_count_reg_delayed_backward.argtypes = [_P, _P, _P, _P, _I, _I, _P, _I, _I, _PP, _P, _P, _P,
                                                         ctypes.c_double, ctypes.c_double, ctypes.c_double, _P, _P,
                                                         _P, _P, _P, _P, _SZ, _P]
    lib.lif_delay_queues_workspace_size.restype = _SZ
    lib.lif_delay_queues_workspace_size.argtypes = [_I, _I, _I]
    lib.lif_delay_queues.restype = _I
    lib.lif_delay_queues.argtypes = [_P, _P, _P, _I, _I, _P, _I, _I, _P, _P, _P, _P, _SZ, _P]
    for name in ("lif_layer_forward_delayed", "lif_layer_forward_delayed_sequential"):
        f = getattr(lib, name)
        f.restype = _I
        f.argtypes = [_P, _P, _P, _P, _I, _I, _P, _I, _I, _PP, _P, _P, _P, _P, _P, _P]
    lib.lif_layer_backward_delayed_workspace_size.restype = _SZ
    lib.lif_layer_backward_delayed_workspace_size.argtypes = [_I, _I, _I, _I, _PP]
    lib.lif_layer_backward_delayed.restype = _I
    lib.lif_layer_backward_delayed.argtypes = [_P, _P, _P, _P, _I, _I, _P, _I, _I, _PP, _P, _P, _P, _P, _P, _P, _P,
                                               _P, _P, _SZ, _P]
    lib.lif_add.restype = _I
    lib.lif_add.argtypes = [_P, _P, _SZ, _P]
    lib.lif_softplus.restype = _I
    lib.lif_softplus.argtypes = [_P, _P, _SZ, ctypes.c_double, _P]
    lib.lif_softplus_grad.restype = _I
    lib.lif_softplus_grad.argtypes = [_P, _P, _P, _SZ, ctypes.c_double, _P]
    lib.lif_timer_enable.restype = None
    lib.lif_timer_enable.argtypes = [_I]
    lib.lif_timer_read.restype = _I
    lib.lif_timer_read.argtypes = [ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_double),
                                   ctypes.POINTER(ctypes.c_int32), _I]
    _lib = lib
    return lib


# ---------------------------------------------------------------------------
# C entry points under their own names (raw pointers / ints)
# ---------------------------------------------------------------------------

def lif_version() -> str:
    return load().lif_version().decode()


def lif_layer_forward_workspace_size(B, E_max, C_in, N_out, p: lif_params) -> int:
    return int(load().lif_layer_forward_workspace_size(B, E_max, C_in, N_out, ctypes.byref(p)))


def lif_layer_backward_workspace_size(B, E_max, C_in, N_out, p: lif_params) -> int:
    return int(load().lif_layer_backward_workspace_size(B, E_max, C_in, N_out, ctypes.byref(p)))


def lif_merge_workspace_size(B, N, s_max, E2_max) -> int:
    return int(load().lif_merge_workspace_size(B, N, s_max, E2_max))


def lif_layer_forward(*args) -> int:
    return load().lif_layer_forward(*args)


def lif_layer_forward_sequential(*args) -> int:
    return load().lif_layer_forward_sequential(*args)


def lif_layer_forward_chunked(*args) -> int:
    return load().lif_layer_forward_chunked(*args)


def lif_layer_forward_noalloc(*args) -> int:
    return load().lif_layer_forward_noalloc(*args)


def lif_layer_forward_noalloc_max_bytes() -> int:
    return int(load().lif_layer_forward_noalloc_max_bytes())


def lif_layer_backward(*args) -> int:
    return load().lif_layer_backward(*args)


def lif_merge_spikes(*args) -> int:
    return load().lif_merge_spikes(*args)


def lif_merge_grad(*args) -> int:
    return load().lif_merge_grad(*args)


def lif_li_readout_workspace_size(B, E_max, C_in, N_cls) -> int:
    return int(load().lif_li_readout_workspace_size(B, E_max, C_in, N_cls))


def lif_li_readout(*args) -> int:
    return load().lif_li_readout(*args)


def lif_spike_count_reg_workspace_size(B, E_max, C_in, N_out) -> int:
    return int(load().lif_spike_count_reg_workspace_size(B, E_max, C_in, N_out))


def lif_spike_count_reg(*args) -> int:
    return load().lif_spike_count_reg(*args)


def lif_adam_step(*args) -> int:
    return load().lif_adam_step(*args)


def lif_first_spike_ce(*args) -> int:
    return load().lif_first_spike_ce(*args)


def lif_spike_count_reg_backward_workspace_size(B, E_max, C_in, N_out) -> int:
    return load().lif_spike_count_reg_backward_workspace_size(B, E_max, C_in, N_out)


def lif_spike_count_reg_backward(*args) -> int:
    return load().lif_spike_count_reg_backward(*args)


def lif_delay_queues_workspace_size(B, E_max, N_out) -> int:
    return load().lif_delay_queues_workspace_size(B, E_max, N_out)


def lif_delay_queues(*args) -> int:
    return load().lif_delay_queues(*args)


def lif_layer_forward_delayed(*args) -> int:
    return load().lif_layer_forward_delayed(*args)


def lif_layer_forward_delayed_sequential(*args) -> int:
    return load().lif_layer_forward_delayed_sequential(*args)


def lif_layer_backward_delayed_workspace_size(B, E_max, C_in, N_out, p: lif_params) -> int:
    return load().lif_layer_backward_delayed_workspace_size(B, E_max, C_in, N_out, ctypes.byref(p))


def lif_layer_backward_delayed(*args) -> int:
    return load().lif_layer_backward_delayed(*args)


def lif_spike_count_reg_delayed_workspace_size(B, E_max, C_in, N_out) -> int:
    return load().lif_spike_count_reg_delayed_workspace_size(B, E_max, C_in, N_out)


def lif_spike_count_reg_delayed(*args) -> int:
    return load().lif_spike_count_reg_delayed(*args)


def lif_spike_count_reg_delayed_backward(*args) -> int:
    return load().lif_spike_count_reg_delayed_backward(*args)


def lif_add(*args) -> int:
    return load().lif_add(*args)


def lif_softplus(*args) -> int:
    return load().lif_softplus(*args)


def lif_softplus_grad(*args) -> int:
    return load().lif_softplus_grad(*args)


def lif_timer_enable(on: bool) -> None:
    load().lif_timer_enable(1 if on else 0)


def lif_timer_read(cap: int = 32):
    names = (ctypes.c_char_p * cap)()
    ms = (ctypes.c_double * cap)()
    cnt = (ctypes.c_int32 * cap)()
    n = load().lif_timer_read(names, ms, cnt, cap)
    return {names[j].decode(): (ms[j], cnt[j]) for j in range(min(n, cap))}


# ---------------------------------------------------------------------------
# torch conveniences
# ---------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> int:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _check(fn: str, rc: int):
    if rc != LIF_OK:
        raise LifError(fn, rc)


def _dev_inputs(ev_t, ev_src, ev_n, WT):
    torch = _torch()
    for name, t, dt in (("ev_t", ev_t, torch.float32), ("ev_src", ev_src, torch.int32),
                        ("ev_n", ev_n, torch.int32), ("WT", WT, torch.float32)):
        if t.dtype != dt or not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous {dt} CUDA tensor")
    if ev_t.dim() != 2 or ev_src.shape != ev_t.shape or ev_n.dim() != 1 or ev_n.shape[0] != ev_t.shape[0]:
        raise ValueError("ev_t/ev_src must be [B, E_max] and ev_n [B]")
    if WT.dim() != 2:
        raise ValueError("WT must be [C_in, N_out]")
    return ev_t.shape[0], ev_t.shape[1], WT.shape[0], WT.shape[1]


@dataclass
class ForwardOut:
    out_t: "object"     # float32 [B, N, s_max]
    out_n: "object"     # int32 [B, N]
    out_i: "object"     # float32 [B, N, s_max]
    status: "object"    # int32 [LIF_STATUS_WORDS]
    out_k: "object" = None   # int32 [B, N, s_max]: input events consumed before each spike
    queues: "object" = None  # the per-neuron queues of a layer with delays (DelayQueues), else None


def forward(ev_t, ev_src, ev_n, WT, params: Params = Params(), sequential: bool = False, stream=None,
            ws=None, out: Optional[ForwardOut] = None) -> ForwardOut:
    """Run lif_layer_forward (or the sequential baseline) on device tensors."""
    torch = _torch()
    B, E, C, N = _dev_inputs(ev_t, ev_src, ev_n, WT)
    p = params.c()
    dev = ev_t.device
    if out is None:
        out = ForwardOut(torch.empty((B, N, params.s_max), dtype=torch.float32, device=dev),
                         torch.empty((B, N), dtype=torch.int32, device=dev),
                         torch.empty((B, N, params.s_max), dtype=torch.float32, device=dev),
                         torch.empty(LIF_STATUS_WORDS, dtype=torch.int32, device=dev),
                         torch.empty((B, N, params.s_max), dtype=torch.int32, device=dev))
    need = lif_layer_forward_workspace_size(B, E, C, N, p)
    if ws is None or ws.numel() < need:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    fn = lif_layer_forward_sequential if sequential else lif_layer_forward
    rc = fn(_ptr(ev_t), _ptr(ev_src), _ptr(ev_n), B, E, _ptr(WT), C, N, ctypes.byref(p), _ptr(out.out_t),
            _ptr(out.out_n), _ptr(out.out_i), _ptr(out.out_k), _ptr(out.status), _ptr(ws), ws.numel(),
            _stream(stream))
    _check(fn.__name__, rc)
    return out


def backward(ev_t, ev_src, ev_n, WT, fwd: ForwardOut, grad_out_t, params: Params = Params(), stream=None,
             want_time_grad: bool = True, ws=None):
    """Run lif_layer_backward; returns (grad_WT, grad_ev_t or None)."""
    torch = _torch()
    B, E, C, N = _dev_inputs(ev_t, ev_src, ev_n, WT)
    p = params.c()
    dev = ev_t.device
    gW = torch.empty((C, N), dtype=torch.float32, device=dev)
    gT = torch.empty((B, E), dtype=torch.float32, device=dev) if want_time_grad else None
    need = lif_layer_backward_workspace_size(B, E, C, N, p)
    if ws is None or ws.numel() < need:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    g = grad_out_t.contiguous().to(torch.float32)
    rc = lif_layer_backward(_ptr(ev_t), _ptr(ev_src), _ptr(ev_n), B, E, _ptr(WT), C, N, ctypes.byref(p),
                            _ptr(fwd.out_t), _ptr(fwd.out_n), _ptr(fwd.out_i), _ptr(fwd.out_k), _ptr(g), _ptr(gW),
                            _ptr(gT), _ptr(ws), ws.numel(), _stream(stream))
    _check("lif_layer_backward", rc)
    return gW, gT


def merge(fwd: ForwardOut, E2_max: int, stream=None):
    """Run lif_merge_spikes; returns (ev_t2, ev_src2, ev_n2, perm, status)."""
    torch = _torch()
    B, N, S = fwd.out_t.shape
    dev = fwd.out_t.device
    ev_t2 = torch.empty((B, E2_max), dtype=torch.float32, device=dev)
    ev_src2 = torch.empty((B, E2_max), dtype=torch.int32, device=dev)
    ev_n2 = torch.empty(B, dtype=torch.int32, device=dev)
    perm = torch.empty((B, E2_max), dtype=torch.int32, device=dev)
    status = torch.empty(LIF_STATUS_WORDS, dtype=torch.int32, device=dev)
    need = lif_merge_workspace_size(B, N, S, E2_max)
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    rc = lif_merge_spikes(_ptr(fwd.out_t), _ptr(fwd.out_n), B, N, S, _ptr(ev_t2), _ptr(ev_src2), _ptr(ev_n2),
                          _ptr(perm), E2_max, _ptr(status), _ptr(ws), ws.numel(), _stream(stream))
    _check("lif_merge_spikes", rc)
    return ev_t2, ev_src2, ev_n2, perm, status


def first_spike_ce(fwd: ForwardOut, labels, tau0: float, t_silent: float, stream=None):
    """Run lif_first_spike_ce; returns (loss [1], grad_out_t [B, N, s_max])."""
    torch = _torch()
    B, N, S = fwd.out_t.shape
    dev = fwd.out_t.device
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    g = torch.empty((B, N, S), dtype=torch.float32, device=dev)
    lab = labels.to(device=dev, dtype=torch.int32).contiguous()
    rc = lif_first_spike_ce(_ptr(fwd.out_t), _ptr(fwd.out_n), B, N, S, _ptr(lab), float(tau0), float(t_silent),
                            _ptr(loss), _ptr(g), _stream(stream))
    _check("lif_first_spike_ce", rc)
    return loss, g


def merge_grad(grad_ev_t2, perm, ev_n2, N: int, s_max: int, stream=None):
    """Run lif_merge_grad; returns grad_out_t [B, N, s_max]."""
    torch = _torch()
    B, E2 = grad_ev_t2.shape
    g = torch.empty((B, N, s_max), dtype=torch.float32, device=grad_ev_t2.device)
    rc = lif_merge_grad(_ptr(grad_ev_t2), _ptr(perm), _ptr(ev_n2), B, E2, N, s_max, _ptr(g), _stream(stream))
    _check("lif_merge_grad", rc)
    return g


def li_readout(ev_t, ev_src, ev_n, WT, q: LiParams = LiParams(), labels=None, grads: bool = True, stream=None,
               ws=None):
    """Run lif_li_readout; returns (logits [B, N_cls], loss [1] or None,
    grad_WT or None, grad_ev_t or None)."""
    torch = _torch()
    B, E, C, K = _dev_inputs(ev_t, ev_src, ev_n, WT)
    dev = ev_t.device
    logits = torch.empty((B, K), dtype=torch.float32, device=dev)
    loss = gW = gT = lab = None
    if labels is not None:
        lab = labels.to(device=dev, dtype=torch.int32).contiguous()
        loss = torch.empty(1, dtype=torch.float32, device=dev)
        if grads:
            gW = torch.empty((C, K), dtype=torch.float32, device=dev)
            gT = torch.empty((B, E), dtype=torch.float32, device=dev)
    need = lif_li_readout_workspace_size(B, E, C, K)
    if ws is None or ws.numel() < need:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    qc = q.c()
    rc = lif_li_readout(_ptr(ev_t), _ptr(ev_src), _ptr(ev_n), B, E, _ptr(WT), C, K, ctypes.byref(qc), _ptr(lab),
                        _ptr(logits), _ptr(loss), _ptr(gW), _ptr(gT), _ptr(ws), ws.numel(), _stream(stream))
    _check("lif_li_readout", rc)
    return logits, loss, gW, gT


def adam_step(param, grad, m1, m2, step: int, lr: float = 1e-3, beta1: float = 0.9, beta2: float = 0.999,
              eps: float = 1e-8, stream=None):
    """Run lif_adam_step on contiguous float32 tensors of one shape (in place)."""
    for t in (param, grad, m1, m2):
        if not t.is_contiguous() or t.numel() != param.numel():
            raise ValueError("adam_step needs contiguous tensors of one size")
    a = lif_adam_params(lr, beta1, beta2, eps)
    rc = lif_adam_step(_ptr(param), _ptr(grad), _ptr(m1), _ptr(m2), param.numel(), ctypes.byref(a), int(step),
                       _stream(stream))
    _check("lif_adam_step", rc)


def spike_count_reg(ev_t, ev_src, ev_n, WT, fwd: ForwardOut, c_target: float, params: Params = Params(),
                    stream=None, ws=None):
    """Run lif_spike_count_reg; returns (loss [2] = (L_reg, L_over), under
    [B, N], over [B, N])."""
    torch = _torch()
    B, E, C, N = _dev_inputs(ev_t, ev_src, ev_n, WT)
    dev = ev_t.device
    loss = torch.empty(2, dtype=torch.float32, device=dev)
    under = torch.empty((B, N), dtype=torch.float32, device=dev)
    over = torch.empty((B, N), dtype=torch.float32, device=dev)
    need = lif_spike_count_reg_workspace_size(B, E, C, N)
    if ws is None or ws.numel() < need:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    p = params.c()
    rc = lif_spike_count_reg(_ptr(ev_t), _ptr(ev_src), _ptr(ev_n), B, E, _ptr(WT), C, N, ctypes.byref(p),
                             _ptr(fwd.out_t), _ptr(fwd.out_n), _ptr(fwd.out_k), float(c_target), _ptr(loss),
                             _ptr(under), _ptr(over), _ptr(ws), ws.numel(), _stream(stream))
    _check("lif_spike_count_reg", rc)
    return loss, under, over


def forward_chunked(ev_t, ev_src, ev_n, WT, K: int = 128, C: int = 0, params: Params = Params(), stream=None):
    """Run lif_layer_forward_chunked; returns (ForwardOut, consumed [B, N],
    processed [B, N])."""
    torch = _torch()
    B, E, Cin, N = _dev_inputs(ev_t, ev_src, ev_n, WT)
    dev = ev_t.device
    p = params.c()
    out = ForwardOut(torch.empty((B, N, params.s_max), dtype=torch.float32, device=dev),
                     torch.empty((B, N), dtype=torch.int32, device=dev),
                     torch.empty((B, N, params.s_max), dtype=torch.float32, device=dev),
                     torch.empty(LIF_STATUS_WORDS, dtype=torch.int32, device=dev),
                     torch.empty((B, N, params.s_max), dtype=torch.int32, device=dev))
    consumed = torch.empty((B, N), dtype=torch.int32, device=dev)
    processed = torch.empty((B, N), dtype=torch.int32, device=dev)
    rc = lif_layer_forward_chunked(_ptr(ev_t), _ptr(ev_src), _ptr(ev_n), B, E, _ptr(WT), Cin, N, ctypes.byref(p),
                                   int(K), int(C), _ptr(out.out_t), _ptr(out.out_n), _ptr(out.out_i),
                                   _ptr(out.out_k), _ptr(consumed), _ptr(processed), _ptr(out.status),
                                   _stream(stream))
    _check("lif_layer_forward_chunked", rc)
    return out, consumed, processed


@dataclass
class DelayQueues:
    q_t: "object"       # float32 [B, N, E_max]: arrival times, each neuron's queue in order
    q_k: "object"       # int32 [B, N, E_max]: the sample's event index of each entry
    status: "object"    # int32 [LIF_STATUS_WORDS]


def delay_queues(ev_t, ev_src, ev_n, DT, stream=None, ws=None) -> DelayQueues:
    """Run lif_delay_queues: each neuron's queue of arrivals t_k + DT[src_k, i]."""
    torch = _torch()
    B, E, C, N = _dev_inputs(ev_t, ev_src, ev_n, DT)
    dev = ev_t.device
    q = DelayQueues(torch.empty((B, N, E), dtype=torch.float32, device=dev),
                    torch.empty((B, N, E), dtype=torch.int32, device=dev),
                    torch.empty(LIF_STATUS_WORDS, dtype=torch.int32, device=dev))
    need = lif_delay_queues_workspace_size(B, E, N)
    if ws is None or ws.numel() < need:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    rc = lif_delay_queues(_ptr(ev_t), _ptr(ev_src), _ptr(ev_n), B, E, _ptr(DT), C, N, _ptr(q.q_t), _ptr(q.q_k),
                          _ptr(q.status), _ptr(ws), ws.numel(), _stream(stream))
    _check("lif_delay_queues", rc)
    return q


def _queue_inputs(q: DelayQueues, ev_src, ev_n, WT):
    torch = _torch()
    B, E, C, N = _dev_inputs(q.q_t.new_empty(ev_src.shape), ev_src, ev_n, WT)
    for name, t, dt in (("q_t", q.q_t, torch.float32), ("q_k", q.q_k, torch.int32)):
        if t.dtype != dt or not t.is_cuda or not t.is_contiguous() or tuple(t.shape) != (B, N, E):
            raise ValueError(f"{name} must be a contiguous {dt} CUDA tensor [B, N_out, E_max]")
    return B, E, C, N


def forward_delayed(q: DelayQueues, ev_src, ev_n, WT, params: Params = Params(), sequential: bool = False,
                    stream=None) -> ForwardOut:
    """Run lif_layer_forward_delayed (or its sequential baseline) on the
    queues of delay_queues."""
    torch = _torch()
    B, E, C, N = _queue_inputs(q, ev_src, ev_n, WT)
    dev = WT.device
    p = params.c()
    out = ForwardOut(torch.empty((B, N, params.s_max), dtype=torch.float32, device=dev),
                     torch.empty((B, N), dtype=torch.int32, device=dev),
                     torch.empty((B, N, params.s_max), dtype=torch.float32, device=dev),
                     torch.empty(LIF_STATUS_WORDS, dtype=torch.int32, device=dev),
                     torch.empty((B, N, params.s_max), dtype=torch.int32, device=dev))
    fn = lif_layer_forward_delayed_sequential if sequential else lif_layer_forward_delayed
    rc = fn(_ptr(q.q_t), _ptr(q.q_k), _ptr(ev_src), _ptr(ev_n), B, E, _ptr(WT), C, N, ctypes.byref(p),
            _ptr(out.out_t), _ptr(out.out_n), _ptr(out.out_i), _ptr(out.out_k), _ptr(out.status), _stream(stream))
    _check(fn.__name__, rc)
    return out


def backward_delayed(q: DelayQueues, ev_src, ev_n, WT, fwd: ForwardOut, grad_out_t, params: Params = Params(),
                     stream=None, want_delay_grad: bool = True, want_time_grad: bool = True, ws=None):
    """Run lif_layer_backward_delayed; returns (grad_WT, grad_DT or None,
    grad_ev_t or None)."""
    torch = _torch()
    B, E, C, N = _queue_inputs(q, ev_src, ev_n, WT)
    dev = WT.device
    p = params.c()
    gW = torch.empty((C, N), dtype=torch.float32, device=dev)
    gD = torch.empty((C, N), dtype=torch.float32, device=dev) if want_delay_grad else None
    gT = torch.empty((B, E), dtype=torch.float32, device=dev) if want_time_grad else None
    need = lif_layer_backward_delayed_workspace_size(B, E, C, N, p)
    if not want_time_grad:
        need -= B * N * E * 8          # no per-event dL/dt terms are stored
    if ws is None or ws.numel() < need:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    g = grad_out_t.contiguous().to(torch.float32)
    rc = lif_layer_backward_delayed(_ptr(q.q_t), _ptr(q.q_k), _ptr(ev_src), _ptr(ev_n), B, E, _ptr(WT), C, N,
                                    ctypes.byref(p), _ptr(fwd.out_t), _ptr(fwd.out_n), _ptr(fwd.out_i),
                                    _ptr(fwd.out_k), _ptr(g), _ptr(gW), _ptr(gD), _ptr(gT), _ptr(ws), ws.numel(),
                                    _stream(stream))
    _check("lif_layer_backward_delayed", rc)
    return gW, gD, gT


def spike_count_reg_backward(ev_t, ev_src, ev_n, WT, fwd: ForwardOut, c_target: float, lam_reg: float = 1.0,
                             lam_over: float = 1.0, params: Params = Params(), grad_spike=None,
                             want_time_grad: bool = True, stream=None, ws=None):
    """Run lif_spike_count_reg_backward; returns (loss [2], grad_spike
    [B, N, s_max] (the given tensor, added to, or a new one), direct grad_WT,
    direct grad_ev_t or None)."""
    torch = _torch()
    B, E, C, N = _dev_inputs(ev_t, ev_src, ev_n, WT)
    dev = ev_t.device
    p = params.c()
    loss = torch.empty(2, dtype=torch.float32, device=dev)
    if grad_spike is None:
        grad_spike = torch.zeros((B, N, params.s_max), dtype=torch.float32, device=dev)
    gW = torch.empty((C, N), dtype=torch.float32, device=dev)
    gT = torch.empty((B, E), dtype=torch.float32, device=dev) if want_time_grad else None
    need = lif_spike_count_reg_backward_workspace_size(B, E, C, N)
    if ws is None or ws.numel() < need:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    rc = lif_spike_count_reg_backward(_ptr(ev_t), _ptr(ev_src), _ptr(ev_n), B, E, _ptr(WT), C, N, ctypes.byref(p),
                                      _ptr(fwd.out_t), _ptr(fwd.out_n), _ptr(fwd.out_k), float(c_target),
                                      float(lam_reg), float(lam_over), _ptr(loss), _ptr(grad_spike), _ptr(gW),
                                      _ptr(gT), _ptr(ws), ws.numel(), _stream(stream))
    _check("lif_spike_count_reg_backward", rc)
    return loss, grad_spike, gW, gT


def spike_count_reg_delayed(q: DelayQueues, ev_src, ev_n, WT, fwd: ForwardOut, c_target: float,
                            params: Params = Params(), stream=None, ws=None):
    """Run lif_spike_count_reg_delayed on the queues of delay_queues and the
    delayed forward's outputs; returns (loss [2], under [B, N], over [B, N])."""
    torch = _torch()
    B, E, C, N = _queue_inputs(q, ev_src, ev_n, WT)
    dev = WT.device
    p = params.c()
    loss = torch.empty(2, dtype=torch.float32, device=dev)
    under = torch.empty((B, N), dtype=torch.float32, device=dev)
    over = torch.empty((B, N), dtype=torch.float32, device=dev)
    need = lif_spike_count_reg_delayed_workspace_size(B, E, C, N)
    if ws is None or ws.numel() < need:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    rc = lif_spike_count_reg_delayed(_ptr(q.q_t), _ptr(q.q_k), _ptr(ev_src), _ptr(ev_n), B, E, _ptr(WT), C, N,
                                     ctypes.byref(p), _ptr(fwd.out_t), _ptr(fwd.out_n), _ptr(fwd.out_k),
                                     float(c_target), _ptr(loss), _ptr(under), _ptr(over), _ptr(ws), ws.numel(),
                                     _stream(stream))
    _check("lif_spike_count_reg_delayed", rc)
    return loss, under, over


def spike_count_reg_delayed_backward(q: DelayQueues, ev_src, ev_n, WT, fwd: ForwardOut, c_target: float,
                                     lam_reg: float = 1.0, lam_over: float = 1.0, params: Params = Params(),
                                     grad_spike=None, want_delay_grad: bool = True, want_time_grad: bool = True,
                                     stream=None, ws=None):
    """Run lif_spike_count_reg_delayed_backward; returns (loss [2],
    grad_spike [B, N, s_max] (the given tensor, added to, or a new one),
    direct grad_WT, direct grad_DT or None, direct grad_ev_t or None)."""
    torch = _torch()
    B, E, C, N = _queue_inputs(q, ev_src, ev_n, WT)
    dev = WT.device
    p = params.c()
    loss = torch.empty(2, dtype=torch.float32, device=dev)
    if grad_spike is None:
        grad_spike = torch.zeros((B, N, params.s_max), dtype=torch.float32, device=dev)
    gW = torch.empty((C, N), dtype=torch.float32, device=dev)
    gD = torch.empty((C, N), dtype=torch.float32, device=dev) if want_delay_grad else None
    gT = torch.empty((B, E), dtype=torch.float32, device=dev) if want_time_grad else None
    need = lif_spike_count_reg_delayed_workspace_size(B, E, C, N)
    if ws is None or ws.numel() < need:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    rc = lif_spike_count_reg_delayed_backward(_ptr(q.q_t), _ptr(q.q_k), _ptr(ev_src), _ptr(ev_n), B, E, _ptr(WT), C,
                                              N, ctypes.byref(p), _ptr(fwd.out_t), _ptr(fwd.out_n), _ptr(fwd.out_k),
                                              float(c_target), float(lam_reg), float(lam_over), _ptr(loss),
                                              _ptr(grad_spike), _ptr(gW), _ptr(gD), _ptr(gT), _ptr(ws), ws.numel(),
                                              _stream(stream))
    _check("lif_spike_count_reg_delayed_backward", rc)
    return loss, grad_spike, gW, gD, gT


def add_(y, x, stream=None):
    """y += x on the device (lif_add); returns y."""
    if y.shape != x.shape or y.dtype != x.dtype:
        raise ValueError("add_: shapes and dtypes must match")
    _check("lif_add", lif_add(_ptr(y), _ptr(x.contiguous()), y.numel(), _stream(stream)))
    return y


def softplus(x, beta: float, stream=None):
    """d = softplus(x) = log(1 + e^{beta x}) / beta (lif_softplus)."""
    d = _torch().empty_like(x)
    _check("lif_softplus", lif_softplus(_ptr(x), _ptr(d), x.numel(), float(beta), _stream(stream)))
    return d


def softplus_grad(x, grad_d, beta: float, stream=None):
    """grad_x = grad_d * sigmoid(beta x) (lif_softplus_grad)."""
    gx = _torch().empty_like(x)
    _check("lif_softplus_grad", lif_softplus_grad(_ptr(x), _ptr(grad_d), _ptr(gx), x.numel(), float(beta),
                                                  _stream(stream)))
    return gx
