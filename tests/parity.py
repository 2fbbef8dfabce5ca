"""Comparison helpers shared by the GPU parity tests (GPU path vs oracle)."""
from __future__ import annotations

import numpy as np

TIME_RTOL = 1e-5        # spike times: |t_gpu - t_or| <= 1e-5 |t_or|
GRAD_RTOL = 1e-4        # gradients: per-tensor norm and element-wise (floored) relative error
# End to end (GPU forward + backward against the oracle's forward +
# backward) the spike times and the currents at the spikes reach the
# backward pass rounded to float32, as the layer's outputs are.  The oracle
# measures what that rounding does by itself: g_or32, its gradient of its own
# spike train rounded to float32, against g_or, its exact gradient.  In norm
# the two differ by at most ~1e-5; element-wise, entries that are sums of
# large, nearly cancelling terms (a spike close to grazing has a large
# adjoint) move by up to ~2.5e-3 (floored relative, on 20 000-event trains).
# Such an entry is ill-conditioned with respect to the float32 hand-over and
# is compared with g_or32; every other entry with g_or.
COND_RTOL = 1e-5


MAX_EXCUSED_FRAC = 0.01   # at most 1 % of (sample, neuron) pairs may diverge after a near-tie


def _same_train(go, ro, gi, ri, gk=None, rk=None):
    """Float32 GPU spike train go (currents gi) against the oracle's ro (ri):
    same length, times within TIME_RTOL, currents within TIME_RTOL (floored
    at 1e-3), strictly increasing.  Returns (ok, worst time err, worst I err)."""
    if len(go) != len(ro):
        return False, np.inf, np.inf
    if len(ro) == 0:
        return True, 0.0, 0.0
    if gk is not None and not np.array_equal(gk, rk):
        return False, np.inf, np.inf
    et = np.abs(go - ro) / np.abs(ro)
    ei = 0.0
    if gi is not None:
        ei = float((np.abs(gi - ri) / np.maximum(np.abs(ri), 1e-3)).max())
    ok = et.max() <= TIME_RTOL and ei <= TIME_RTOL and np.all(np.diff(go) > 0)
    return bool(ok), float(et.max()), ei


def compare_spikes(out_t_gpu, out_n_gpu, ref, out_i_gpu=None, label="", max_excused=MAX_EXCUSED_FRAC,
                   out_k_gpu=None):
    """Spike counts and order identical per (sample, neuron), times and
    currents at the spikes within 1e-5 relative, the consumed-event count of
    every spike identical (when out_k_gpu is given).  A neuron whose oracle
    trajectory came within 1e-6 of the threshold at some interval maximum is
    flagged (ref.tie_t holds the start of that interval).  A flagged neuron
    is still compared in full; only if its trains differ is it excused after
    the tie (the spikes before the tied interval must then match).  At most
    max_excused of all pairs may be excused.  Returns a dict of statistics,
    which the caller prints."""
    tg = np.asarray(out_t_gpu, dtype=np.float64)
    ng = np.asarray(out_n_gpu)
    ig = None if out_i_gpu is None else np.asarray(out_i_gpu, dtype=np.float64)
    kg = None if out_k_gpu is None else np.asarray(out_k_gpu)
    B, N, S = ref.out_t.shape
    tie = np.isfinite(ref.tie_t)
    worst = 0.0
    worst_i = 0.0
    # ---- neurons without a flagged tie: every slot, vectorised
    nt = ~tie
    bad = np.argwhere(nt & (ng != ref.out_n))
    if len(bad):
        b, i = bad[0]
        raise AssertionError(f"{label} count mismatch at (b={b}, i={i}): gpu {ng[b, i]} oracle {ref.out_n[b, i]}")
    slot = np.arange(S)[None, None, :]
    valid = (slot < ref.out_n[..., None]) & nt[..., None]
    if valid.any():
        ro = ref.out_t[valid]
        err = np.abs(tg[valid] - ro) / np.abs(ro)
        worst = float(err.max())
        if worst > TIME_RTOL:
            b, i, s = np.argwhere(valid)[int(err.argmax())]
            raise AssertionError(f"{label} time mismatch at ({b},{i}) spike {s}: {tg[b, i, s]} vs {ref.out_t[b, i, s]}")
        later = valid[..., 1:]
        assert np.all(tg[..., 1:][later] > tg[..., :-1][later]), f"{label} spike order"
        if kg is not None:
            bad = np.argwhere(valid & (kg != ref.out_k))
            assert len(bad) == 0, f"{label} consumed-event count differs at {tuple(bad[0])}"
        if ig is not None:
            ri = ref.out_i[valid]
            e = np.abs(ig[valid] - ri) / np.maximum(np.abs(ri), 1e-3)
            worst_i = float(e.max())
            assert worst_i <= TIME_RTOL, f"{label} I* mismatch (worst {worst_i:.3e})"
    pad = (slot >= ref.out_n[..., None]) & nt[..., None]
    assert np.all(np.isinf(tg[pad])), f"{label} padding"
    if kg is not None:
        assert np.all(kg[pad] == 0), f"{label} padding of out_k"
    # ---- flagged neurons: in full if the trains agree, else before the tie
    excused = 0
    excused_pairs = []
    for b, i in np.argwhere(tie):
        nr, n_g = int(ref.out_n[b, i]), int(ng[b, i])
        go, ro = tg[b, i, :n_g], ref.out_t[b, i, :nr]
        gi = None if ig is None else ig[b, i, :n_g]
        ri = ref.out_i[b, i, :nr]
        gk = None if kg is None else kg[b, i, :n_g]
        ok, et, ei = _same_train(go, ro, gi, ri, gk, ref.out_k[b, i, :nr])
        if ok:
            worst, worst_i = max(worst, et), max(worst_i, ei)
            continue
        excused += 1
        excused_pairs.append((int(b), int(i)))
        t_tie = ref.tie_t[b, i]
        kr, kg_ = int((ro < t_tie).sum()), int((go < t_tie).sum())
        ok, et, ei = _same_train(go[:kg_], ro[:kr], None if gi is None else gi[:kg_], ri[:kr],
                                 None if gk is None else gk[:kg_], ref.out_k[b, i, :kr])
        assert ok, f"{label} spikes before a tie at (b={b}, i={i}) differ: {go[:kg_]} vs {ro[:kr]}"
        worst, worst_i = max(worst, et), max(worst_i, ei)
    frac = excused / float(B * N)
    assert frac <= max_excused, f"{label}: {excused} of {B * N} neurons diverge after a near-tie ({frac:.2%})"
    return {"flagged": int(tie.sum()), "excused": excused, "compared": int(B * N), "worst_time_rel": worst,
            "worst_i_rel": worst_i, "spikes": int(ref.out_n.sum()), "excused_pairs": excused_pairs}


def compare_grad(g_gpu, g_or, mask=None, label="", elem_rtol=GRAD_RTOL):
    g_gpu = np.asarray(g_gpu, dtype=np.float64)
    g_or = np.asarray(g_or, dtype=np.float64)
    if mask is not None:
        g_gpu = g_gpu[mask]
        g_or = g_or[mask]
    nrm = np.linalg.norm(g_or)
    if nrm == 0:
        assert np.all(g_gpu == 0), f"{label}: oracle gradient is zero, GPU's is not"
        return 0.0
    rel = np.linalg.norm(g_gpu - g_or) / nrm
    assert rel <= GRAD_RTOL, f"{label}: norm-wise relative error {rel:.3e}"
    floor = 1e-3 * np.abs(g_or).max()
    el = np.abs(g_gpu - g_or) / np.maximum(np.abs(g_or), floor)
    assert el.max() <= elem_rtol, f"{label}: element-wise relative error {el.max():.3e}"
    return float(rel)


def compare_grad_e2e(g_gpu, g_or, g_or32, label=""):
    """End-to-end gradient check (see COND_RTOL): norm-wise against g_or;
    element-wise against g_or where the float32 hand-over moves the oracle's
    own gradient by at most COND_RTOL (floored relative), against g_or32
    elsewhere.  Returns (norm-wise relative error, ill-conditioned fraction)."""
    g_gpu = np.asarray(g_gpu, dtype=np.float64)
    g_or = np.asarray(g_or, dtype=np.float64)
    g_or32 = np.asarray(g_or32, dtype=np.float64)
    nrm = np.linalg.norm(g_or)
    if nrm == 0:
        assert np.all(g_gpu == 0), f"{label}: oracle gradient is zero, GPU's is not"
        return 0.0, 0.0
    rel = float(np.linalg.norm(g_gpu - g_or) / nrm)
    assert rel <= GRAD_RTOL, f"{label}: norm-wise relative error {rel:.3e}"
    den = np.maximum(np.abs(g_or), 1e-3 * np.abs(g_or).max())
    ill = np.abs(g_or32 - g_or) / den > COND_RTOL
    e = np.abs(g_gpu - g_or) / den
    if (~ill).any():
        w = float(e[~ill].max())
        assert w <= GRAD_RTOL, f"{label}: element-wise relative error {w:.3e} (well-conditioned entries)"
    if ill.any():
        den32 = np.maximum(np.abs(g_or32), 1e-3 * np.abs(g_or32).max())
        w = float((np.abs(g_gpu - g_or32) / den32)[ill].max())
        assert w <= GRAD_RTOL, f"{label}: element-wise relative error {w:.3e} against the float32 hand-over"
    return rel, float(ill.mean())


def compare_grad_band(g_gpu, g_or, g_or64, label=""):
    """Regulariser gradient check on a spike train handed over in float32:
    norm-wise and element-wise (floored) against g_or, the oracle at those
    float32 spike times, except where the rounding of the hand-over itself
    moves the oracle's gradient (g_or64: at its exact spike times) by more
    than COND_RTOL; there the element must lie within GRAD_RTOL of the band
    between g_or and g_or64.  The GPU takes the reset of a spike at a float32
    time as the decaying deficit of a threshold crossing there, the oracle as
    V set to V_reset there; the two agree to that rounding, to which such an
    element is sensitive.  Returns (norm-wise error, ill-conditioned
    fraction)."""
    g_gpu = np.asarray(g_gpu, dtype=np.float64)
    g_or = np.asarray(g_or, dtype=np.float64)
    g_or64 = np.asarray(g_or64, dtype=np.float64)
    nrm = np.linalg.norm(g_or)
    if nrm == 0:
        assert np.all(g_gpu == 0), f"{label}: oracle gradient is zero, GPU's is not"
        return 0.0, 0.0
    rel = float(np.linalg.norm(g_gpu - g_or) / nrm)
    assert rel <= GRAD_RTOL, f"{label}: norm-wise relative error {rel:.3e}"
    den = np.maximum(np.abs(g_or), 1e-3 * np.abs(g_or).max())
    ill = np.abs(g_or64 - g_or) / den > COND_RTOL
    e = np.abs(g_gpu - g_or) / den
    if (~ill).any():
        w = float(e[~ill].max())
        assert w <= GRAD_RTOL, f"{label}: element-wise relative error {w:.3e} (well-conditioned entries)"
    if ill.any():
        lo, hi = np.minimum(g_or, g_or64), np.maximum(g_or, g_or64)
        out = np.maximum(lo - g_gpu, 0.0) + np.maximum(g_gpu - hi, 0.0)
        w = float((out / den)[ill].max())
        assert w <= GRAD_RTOL, f"{label}: element-wise relative error {w:.3e} outside the hand-over band"
    return rel, float(ill.mean())
