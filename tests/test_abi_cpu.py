"""Host-side checks of the C ABI (no GPU needed): every symbol declared in
include/lif.h is exported by liblif.so, and argument errors are rejected on
the host before any launch."""
import ctypes
import math
import os
import re

import pytest

import paper_2603_13283_amd as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
F = ctypes.c_void_p(0x1000)      # never dereferenced: validation fails first


def declared_symbols():
    txt = open(os.path.join(ROOT, "include", "lif.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(lif_[a-z_]+)\s*\(", txt)))


@pytest.fixture(scope="module")
def lib():
    return L.load()


def test_every_declared_symbol_is_exported(lib):
    names = declared_symbols()
    assert len(names) >= 10
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(L.EXPORTED)


def test_version_and_workspace_sizes(lib):
    assert "gfx950" in L.lif_version()
    p = L.Params().c()
    small = L.lif_layer_forward_workspace_size(1, 10, 4, 8, p)
    big = L.lif_layer_forward_workspace_size(32, 5200, 700, 256, p)
    assert 0 < small < big < 2 ** 31
    assert L.lif_layer_forward_workspace_size(-1, 10, 4, 8, p) == 0
    # the pool's entries per sample enter the workspace size
    p0, p9 = L.Params(pool_cap=0).c(), L.Params(pool_cap=9000).c()
    assert (L.lif_layer_forward_workspace_size(32, 5200, 700, 256, p0)
            < L.lif_layer_forward_workspace_size(32, 5200, 700, 256, p9))
    assert L.lif_layer_backward_workspace_size(4, 100, 10, 20, p) > 0
    assert L.lif_merge_workspace_size(4, 20, 8, 100) > 0


def _fwd(fn, p, B=2, E=10, C=4, N=8, ws_bytes=10 ** 9, null=None):
    # ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, p, out_t, out_n, out_i, out_k, status, ws, ws_bytes, stream
    args = [F, F, F, B, E, F, C, N, ctypes.byref(p), F, F, F, F, F, F, ws_bytes, None]
    if null is not None:
        args[null] = None
    return fn(*args)


@pytest.mark.parametrize("fn", [L.lif_layer_forward, L.lif_layer_forward_sequential])
def test_forward_argument_errors(lib, fn):
    assert _fwd(fn, L.Params(tau_mem=0.005, tau_syn=0.005).c()) == L.LIF_ERR_TAU
    assert _fwd(fn, L.Params(tau_mem=0.005, tau_syn=0.01).c()) == L.LIF_ERR_TAU
    assert _fwd(fn, L.Params(tau_syn=0.0).c()) == L.LIF_ERR_TAU
    assert _fwd(fn, L.Params(v_th=0.0, v_reset=0.0).c()) == L.LIF_ERR_THRESHOLD
    assert _fwd(fn, L.Params(v_th=1.0, v_reset=2.0).c()) == L.LIF_ERR_THRESHOLD
    assert _fwd(fn, L.Params(v_th=-0.5, v_reset=-1.0).c()) == L.LIF_ERR_THRESHOLD
    assert _fwd(fn, L.Params(s_max=0).c()) == L.LIF_ERR_ARG
    assert _fwd(fn, L.Params(t_end=math.nan).c()) == L.LIF_ERR_ARG
    assert _fwd(fn, L.Params(solver_reg=-1.0).c()) == L.LIF_ERR_ARG
    bad = L.Params().c()
    bad.reserved = 1
    assert _fwd(fn, bad) == L.LIF_ERR_ARG
    bad = L.Params().c()
    bad.flags = 8                                   # no such flag
    assert _fwd(fn, bad) == L.LIF_ERR_ARG
    p = L.Params().c()
    assert _fwd(fn, p, B=-1) == L.LIF_ERR_ARG
    assert _fwd(fn, p, N=0) == L.LIF_ERR_ARG
    assert _fwd(fn, p, C=0) == L.LIF_ERR_ARG
    for null in (0, 1, 2, 5, 9, 10, 13, 14):       # ev_t, ev_src, ev_n, WT, out_t, out_n, status, ws
        assert _fwd(fn, p, null=null) == L.LIF_ERR_ARG, null
    assert _fwd(fn, p, ws_bytes=10) == L.LIF_ERR_WORKSPACE
    assert fn(F, F, F, 2, 10, F, 4, 8, None, F, F, F, F, F, F, 10 ** 9, None) == L.LIF_ERR_ARG


def test_backward_and_merge_argument_errors(lib):
    p = L.Params().c()
    # ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, p, out_t, out_n, out_i, out_k, grad_out_t, grad_WT,
    # grad_ev_t, ws, ws_bytes, stream
    base = [F, F, F, 2, 10, F, 4, 8, ctypes.byref(p), F, F, F, F, F, F, F, F, 10 ** 9, None]
    assert L.lif_layer_backward(*base[:11], None, *base[12:]) == L.LIF_ERR_ARG      # out_i required
    assert L.lif_layer_backward(*base[:12], None, *base[13:]) == L.LIF_ERR_ARG      # out_k required
    bad = L.Params(tau_mem=0.001).c()
    assert L.lif_layer_backward(*base[:8], ctypes.byref(bad), *base[9:]) == L.LIF_ERR_TAU
    small = list(base)
    small[17] = 10
    assert L.lif_layer_backward(*small) == L.LIF_ERR_WORKSPACE
    margs = [F, F, 2, 8, 4, F, F, F, F, 100, F, F, 10 ** 6, None]
    m2 = list(margs)
    m2[9] = L.LIF_MERGE_MAX + 1
    assert L.lif_merge_spikes(*m2) == L.LIF_ERR_SIZE
    m3 = list(margs)
    m3[9] = 0
    assert L.lif_merge_spikes(*m3) == L.LIF_ERR_ARG
    assert L.lif_first_spike_ce(F, F, 0, 20, 4, F, 0.02, 1.0, F, F, None) == L.LIF_ERR_ARG
    assert L.lif_first_spike_ce(F, F, 2, 20, 4, F, 0.0, 1.0, F, F, None) == L.LIF_ERR_ARG


def test_library_missing_fails_loudly(tmp_path):
    import importlib
    mod = importlib.import_module("paper_2603_13283_amd")
    saved = mod._lib
    try:
        mod._lib = None
        with pytest.raises(mod.LibraryMissing):
            mod.load(str(tmp_path / "nope.so"))
    finally:
        mod._lib = saved


@pytest.mark.parametrize("fn", [L.lif_layer_forward, L.lif_layer_forward_sequential])
def test_weight_matrix_size_limit(lib, fn):
    """W^T is addressed with 32-bit byte offsets: C_in * N_out must stay below
    2^29 (rejected on the host, forward and backward)."""
    p = L.Params().c()
    assert _fwd(fn, p, C=1 << 15, N=1 << 14) == L.LIF_ERR_SIZE
    assert _fwd(fn, p, C=1 << 15, N=(1 << 14) - 1, ws_bytes=0) == L.LIF_ERR_WORKSPACE
    bargs = [F, F, F, 2, 10, F, 1 << 15, 1 << 14, ctypes.byref(p), F, F, F, F, F, F, F, F, 10 ** 9, None]
    assert L.lif_layer_backward(*bargs) == L.LIF_ERR_SIZE


@pytest.mark.parametrize("B,E,C,N", [(32, 5383, 700, 256), (128, 11429, 700, 512), (64, 20327, 2312, 1024),
                                     (16, 101617, 32768, 2048)])
def test_forward_workspace_formula(lib, B, E, C, N):
    """The forward workspace is the per-(sample, segment, neuron) carried
    state and mask word (16 + 4 bytes), the per-event decays (32 bytes), a
    few per-neuron and per-sample words, and the pool of entering states
    (16 bytes each, a quarter of the dense bound per sample, at most 1 GiB
    in all); every workload of the benchmark fits in 2 GB."""
    p = L.Params().c()
    ws = L.lif_layer_forward_workspace_size(B, E, C, N, p)
    S = -(-E // 64)
    dense = B * S * N * (16 + 4) + B * S * 64 * 32 + B * S * 16 + 2 * B * N * 4 + 2 * B * 32 * 4
    pool = min(B * max(S * 4 * N // 4, 4096) * 16, 1 << 30)
    assert dense + pool <= ws <= dense + pool + 16 * 256
    assert ws <= 2e9


def test_readout_and_merge_grad_argument_errors(lib):
    q = L.LiParams().c()
    ws = 10 ** 9
    # ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_cls, q, labels, logits, loss, grad_WT, grad_ev_t, ws, ws_bytes, stream
    args = [F, F, F, 2, 10, F, 4, 8, ctypes.byref(q), F, F, F, F, F, F, ws, None]

    def call(**kw):
        a = list(args)
        for i, v in kw.items():
            a[int(i[1:])] = v
        return L.lif_li_readout(*a)
    assert call(a7=L.LIF_LI_MAX_CLASSES + 1) == L.LIF_ERR_SIZE
    assert call(a7=0) == L.LIF_ERR_ARG
    assert call(a9=None) == L.LIF_ERR_ARG              # a loss or gradient without labels
    assert call(a14=None) == L.LIF_ERR_ARG             # no workspace
    assert call(a15=10) == L.LIF_ERR_WORKSPACE
    bad = L.LiParams(tau_mem=0.005, tau_syn=0.005).c()
    assert call(a8=ctypes.byref(bad)) == L.LIF_ERR_TAU
    bad = L.LiParams(tau_li=0.0).c()
    assert call(a8=ctypes.byref(bad)) == L.LIF_ERR_TAU
    bad = L.LiParams(tau_max=math.inf).c()
    assert call(a8=ctypes.byref(bad)) == L.LIF_ERR_ARG
    assert L.lif_li_readout_workspace_size(2, 10, 4, 8) > 0
    assert L.lif_merge_grad(F, F, F, 2, 10, 0, 4, F, None) == L.LIF_ERR_ARG
    assert L.lif_merge_grad(F, F, F, 2, 10, 8, 4, None, None) == L.LIF_ERR_ARG


def test_spike_count_reg_argument_errors(lib):
    p = L.Params().c()
    # ev_t, ev_src, ev_n, B, E_max, WT, C_in, N, p, out_t, out_n, out_k, c_target, loss, under, over, ws, ws_bytes, s
    base = [F, F, F, 2, 10, F, 4, 8, ctypes.byref(p), F, F, F, 4.0, F, None, None, F, 10 ** 9, None]

    def call(i, v):
        a = list(base)
        a[i] = v
        return L.lif_spike_count_reg(*a)
    assert call(11, None) == L.LIF_ERR_ARG          # out_k required
    assert call(13, None) == L.LIF_ERR_ARG          # loss required
    assert call(12, 0.0) == L.LIF_ERR_ARG           # c_target > 0
    assert call(17, 10) == L.LIF_ERR_WORKSPACE
    bad = L.Params(tau_mem=0.001).c()
    assert call(8, ctypes.byref(bad)) == L.LIF_ERR_TAU
    assert L.lif_spike_count_reg_workspace_size(2, 10, 4, 8) > 0


def test_delay_argument_errors(lib):
    p = L.Params().c()
    # queues: ev_t, ev_src, ev_n, B, E_max, DT, C_in, N, q_t, q_k, status, ws, ws_bytes, stream
    qb = [F, F, F, 2, 10, F, 4, 8, F, F, None, F, 10 ** 9, None]

    def q(i, v):
        a = list(qb)
        a[i] = v
        return L.lif_delay_queues(*a)
    assert q(5, None) == L.LIF_ERR_ARG              # DT required
    assert q(9, None) == L.LIF_ERR_ARG              # q_k required
    need = L.lif_delay_queues_workspace_size(2, 10, 8)
    assert need >= 2 * 8 * 10 * 4 and q(12, need - 1) == L.LIF_ERR_WORKSPACE
    # queues up to 16384 events are sorted in LDS (arrivals only); longer ones take 64-bit keys as well
    assert 2 * 8 * 16384 * 4 <= L.lif_delay_queues_workspace_size(2, 16384, 8) < 2 * 8 * 16384 * 12
    assert L.lif_delay_queues_workspace_size(2, 16385, 8) >= 2 * 8 * 16385 * 12
    assert L.lif_delay_queues_workspace_size(-1, 10, 8) == 0
    # forward: q_t, q_k, ev_src, ev_n, B, E_max, WT, C_in, N, p, out_t, out_n, out_i, out_k, status, stream
    fb = [F, F, F, F, 2, 10, F, 4, 8, ctypes.byref(p), F, F, F, F, F, None]

    def f(i, v):
        a = list(fb)
        a[i] = v
        return L.lif_layer_forward_delayed(*a)
    assert f(1, None) == L.LIF_ERR_ARG              # q_k required
    assert f(6, None) == L.LIF_ERR_ARG              # WT required
    bad = L.Params(v_th=0.0).c()
    assert f(9, ctypes.byref(bad)) == L.LIF_ERR_THRESHOLD
    # backward: q_t, q_k, ev_src, ev_n, B, E_max, WT, C_in, N, p, out_t, out_n, out_i, out_k, g, gW, gD, gT,
    # ws, ws_bytes, stream
    bb = [F, F, F, F, 2, 10, F, 4, 8, ctypes.byref(p), F, F, F, F, F, F, None, None, F, 10 ** 9, None]

    def b(i, v):
        a = list(bb)
        a[i] = v
        return L.lif_layer_backward_delayed(*a)
    assert b(15, None) == L.LIF_ERR_ARG             # grad_WT required
    assert b(13, None) == L.LIF_ERR_ARG             # out_k required
    need = L.lif_layer_backward_delayed_workspace_size(2, 10, 4, 8, p)
    with_t = list(bb)
    with_t[17], with_t[19] = F, need - 1          # with grad_ev_t: the full size
    assert need > 0 and L.lif_layer_backward_delayed(*with_t) == L.LIF_ERR_WORKSPACE
    # without grad_ev_t the per-event dL/dt terms (B N E_max 8 bytes) are not stored
    assert b(19, need - 2 * 8 * 10 * 8 - 1) == L.LIF_ERR_WORKSPACE
    bad = L.Params(tau_mem=0.001).c()
    assert b(9, ctypes.byref(bad)) == L.LIF_ERR_TAU


def test_spike_count_reg_backward_argument_errors(lib):
    p = L.Params().c()
    # ev_t, ev_src, ev_n, B, E, WT, C, N, p, out_t, out_n, out_k, c_target, lam_reg, lam_over, loss, g_spike, gW, gT,
    # ws, ws_bytes, stream
    base = [F, F, F, 2, 10, F, 4, 8, ctypes.byref(p), F, F, F, 4.0, 1.0, 1.0, None, F, F, None, F, 10 ** 9, None]

    def call(i, v):
        a = list(base)
        a[i] = v
        return L.lif_spike_count_reg_backward(*a)
    assert call(11, None) == L.LIF_ERR_ARG          # out_k required
    assert call(16, None) == L.LIF_ERR_ARG          # grad_spike required
    assert call(17, None) == L.LIF_ERR_ARG          # grad_WT required
    assert call(12, -1.0) == L.LIF_ERR_ARG          # c_target > 0
    assert call(13, math.inf) == L.LIF_ERR_ARG      # finite lambda
    need = L.lif_spike_count_reg_backward_workspace_size(2, 10, 4, 8)
    assert need > L.lif_spike_count_reg_workspace_size(2, 10, 4, 8)
    assert call(20, need - 1) == L.LIF_ERR_WORKSPACE


def test_spike_count_reg_delayed_argument_errors(lib):
    p = L.Params().c()
    # q_t, q_k, ev_src, ev_n, B, E, WT, C, N, p, out_t, out_n, out_k, c_target, loss, under, over, ws, ws_bytes,
    # stream
    fb = [F, F, F, F, 2, 10, F, 4, 8, ctypes.byref(p), F, F, F, 4.0, None, None, None, F, 10 ** 9, None]

    def f(i, v):
        a = list(fb)
        a[i] = v
        return L.lif_spike_count_reg_delayed(*a)
    assert f(1, None) == L.LIF_ERR_ARG              # q_k required
    assert f(12, None) == L.LIF_ERR_ARG             # out_k required
    assert f(13, 0.0) == L.LIF_ERR_ARG              # c_target > 0
    bad = L.Params(v_th=0.0).c()
    assert f(9, ctypes.byref(bad)) == L.LIF_ERR_THRESHOLD
    need = L.lif_spike_count_reg_delayed_workspace_size(2, 10, 4, 8)
    assert need >= 2 * 8 * 11 * 8 and f(18, 256) == L.LIF_ERR_WORKSPACE
    assert L.lif_spike_count_reg_delayed_workspace_size(-1, 10, 4, 8) == 0
    # backward: ... c_target, lam_reg, lam_over, loss, g_spike, gW, gD, gT, ws, ws_bytes, stream
    bb = [F, F, F, F, 2, 10, F, 4, 8, ctypes.byref(p), F, F, F, 4.0, 1.0, 1.0, None, F, F, None, None, F, 10 ** 9,
          None]

    def b(i, v):
        a = list(bb)
        a[i] = v
        return L.lif_spike_count_reg_delayed_backward(*a)
    assert b(17, None) == L.LIF_ERR_ARG             # grad_spike required
    assert b(18, None) == L.LIF_ERR_ARG             # grad_WT required
    assert b(14, math.nan) == L.LIF_ERR_ARG         # finite lambda
    assert b(22, need - 1) == L.LIF_ERR_WORKSPACE
