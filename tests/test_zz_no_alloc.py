"""lif_layer_forward_noalloc (the forward pass with the library's fixed
per-GPU workspace array) against lif_layer_forward with a caller workspace:
identical bits on two calls in a row, the second with a smaller input (the
array keeps the first call's contents)."""
import ctypes

import numpy as np
import pytest

import workloads as W

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


def _noalloc(env, ev, WT, params):
    torch, lif = env
    B, E, C, N = ev.B, ev.E_max, WT.shape[0], WT.shape[1]
    t, s, n, w = (_dev(torch, a) for a in (ev.ev_t, ev.ev_src, ev.ev_n, WT))
    out_t = torch.empty((B, N, params.s_max), dtype=torch.float32, device="cuda:0")
    out_n = torch.empty((B, N), dtype=torch.int32, device="cuda:0")
    out_i = torch.empty((B, N, params.s_max), dtype=torch.float32, device="cuda:0")
    out_k = torch.empty((B, N, params.s_max), dtype=torch.int32, device="cuda:0")
    status = torch.empty(lif.LIF_STATUS_WORDS, dtype=torch.int32, device="cuda:0")
    p = params.c()
    ptr = lambda x: ctypes.c_void_p(x.data_ptr())
    rc = lif.lif_layer_forward_noalloc(ptr(t), ptr(s), ptr(n), B, E, ptr(w), C, N, ctypes.byref(p), ptr(out_t),
                                       ptr(out_n), ptr(out_i), ptr(out_k), ptr(status), None)
    assert rc == 0, rc
    torch.cuda.synchronize()
    return out_t, out_n, out_i, out_k, status


def _same(torch, a, b):
    if a.dtype == torch.float32:
        a, b = a.view(torch.int32), b.view(torch.int32)
    return torch.equal(a, b)


@pytest.mark.parametrize("pool_cap", [-1, 3])
def test_noalloc_matches_forward_twice(env, pool_cap):
    torch, lif = env
    params = lif.Params(s_max=48, pool_cap=pool_cap)
    cases = [W.random_small(41, B=8, C=200, N=256, n_events=3000, T=0.6, gain=12.0),
             W.random_small(42, B=3, C=40, N=70, n_events=500, T=0.3, gain=14.0)]
    for i, cfg in enumerate(cases):
        ev, WT = cfg.events, cfg.layers[0].WT
        print(f"[case] noalloc call {i} B={ev.B} E_max={ev.E_max} N={WT.shape[1]} pool_cap={pool_cap}", flush=True)
        got = _noalloc(env, ev, WT, params)
        ref = lif.forward(*(_dev(torch, a) for a in (ev.ev_t, ev.ev_src, ev.ev_n, WT)), params)
        torch.cuda.synchronize()
        assert int(got[1].sum()) > 0                 # the case has spikes
        for name, a, b in zip(("out_t", "out_n", "out_i", "out_k", "status"), got,
                              (ref.out_t, ref.out_n, ref.out_i, ref.out_k, ref.status)):
            assert _same(torch, a, b), f"call {i}: {name} differs"


def test_noalloc_rejects_oversize(env):
    torch, lif = env
    p = lif.Params().c()
    F = ctypes.c_void_p(0x1000)       # never dereferenced: the size check fails first
    rc = lif.lif_layer_forward_noalloc(F, F, F, 64, 20000, F, 2312, 1024, ctypes.byref(p), F, F, F, F, F, None)
    assert rc == lif.LIF_ERR_SIZE
    assert lif.lif_layer_forward_noalloc_max_bytes() == 64 << 20
