// lif_common.hpp -- device-side model of the current-based LIF neuron used by
// every kernel of the library (gfx950, wave64).
//
// All state arithmetic is float64: on CDNA4 a float64 FMA issues at the same
// per-lane rate as a non-packed float32 FMA, and keeping V and I in float64
// holds the accumulated rounding of streams of 10^4..10^5 events far below
// the 1e-6 threshold band that decides spike counts.  Inputs (times,
// weights) and outputs (spike times, I at spike) are float32.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/lif.h"

namespace lif {

constexpr int kWave = 64;       // CDNA wavefront width
constexpr int kSeg = 128;       // events per scan segment (one wave walks it)
constexpr int kSub = 16;        // events per sub-block (candidate granularity)
constexpr int kSubPerSeg = kSeg / kSub;
static_assert(kSeg % kSub == 0 && kSubPerSeg <= 32, "sub-block mask is 32 bits");

// Model constants derived once on the host from lif_params.
struct Model {
    double tm, ts, th, vr, t_end;
    double kappa;      // tau_s / (tau_m - tau_s)                    (Eq. mem_pot)
    double a_rate;     // 1/tau_s - 1/tau_m                          (Appendix A)
    double c_tv;       // tau_m tau_s / (tau_m - tau_s)               (Eq. t_vmax)
    double inv_tm, inv_ts;
    double t_peak;     // argmax of the unit kernel K(u) = kappa (e^-u/tm - e^-u/ts)
    double th_lo;      // survival threshold of the cheap upper bound (slightly below th)
    double reg;        // backward floor on dV/dt
    int s_max;
    uint32_t flags;
};

// Per-event decay record, shared by every neuron of a sample (the matrix
// M(dt) of Eq. affine depends only on the gap dt to the previous event):
//   A = e^{-dt/tm}, C = kappa (e^{-dt/tm} - e^{-dt/ts}), D = e^{-dt/ts},
//   g = K(min(dt, t_peak)): the largest value the unit kernel reaches inside
//       the gap, used by the no-crossing bound V <= max(V0,0) + max(I0,0) g.
struct alignas(32) Decay {
    double A, C, D, g;
};

// Source channel of an event, clamped into [0, C_in) so that a malformed
// queue can never address outside W (LIF_VALIDATE reports such events).
__device__ __forceinline__ int clamp_src(int s, int C_in) { return min(max(s, 0), C_in - 1); }

// Event count of a sample, clamped into [0, E_max].
__device__ __forceinline__ int clamp_count(int n, int E_max) { return min(max(n, 0), E_max); }

// Unit kernel K(u) = kappa (e^{-u/tm} - e^{-u/ts}) written with expm1 so that
// tiny gaps do not cancel.
__device__ __forceinline__ double unit_kernel(const Model& m, double u, double eA)
{
    return -m.kappa * eA * expm1(-u * m.a_rate);
}

// Closed-form V after time t from (V0, I0) (Appendix A, Eq. mem_pot).
__device__ __forceinline__ double v_after(const Model& m, double V0, double I0, double t)
{
    if (isinf(t)) return 0.0;
    double em = exp(-t * m.inv_tm);
    return V0 * em + I0 * unit_kernel(m, t, em);
}

// Result of the interval rule.
struct Crossing {
    bool hit;      // V reaches th inside (0, len]
    double hi;     // right end of the root bracket, min(t_Vmax, len)
    double vhi;    // V(hi)
};

// Interval rule of Sec. 3.2.2 for an interval of length len (may be +inf)
// starting at (V0, I0); eA = e^{-len/tm}, eD = e^{-len/ts}, vend = V(len).
// A spike occurs iff V(len) >= th, or the maximum (Eq. t_vmax) lies inside
// the interval and V(t_Vmax) >= th.  The maximum exists only if I0 > V0 and
// D = V0 (tm - ts) + I0 ts > 0; it lies before len iff
// I0 tm e^{-len/ts} < D e^{-len/tm} (the log of Eq. t_vmax compared with
// len without evaluating it).  `th` is passed so the scan can use a
// conservative threshold.
__device__ __forceinline__ Crossing interval_rule(const Model& m, double V0, double I0, double len,
                                                  double eA, double eD, double vend, double th)
{
    Crossing c{false, len, vend};
    // If V(len) >= th the crossing lies in (0, len]: V is unimodal, so V < th
    // before the crossing and V >= th from it to len; [0, len] brackets it.
    if (vend >= th) {
        c.hit = true;
        return c;
    }
    double Dd = V0 * (m.tm - m.ts) + I0 * m.ts;
    bool has_max = (I0 > V0) && (Dd > 0.0);
    bool max_inside = has_max && (isinf(len) || I0 * m.tm * eD < Dd * eA);
    if (max_inside) {
        double tv = m.c_tv * log(I0 * m.tm / Dd);
        if (tv < len) {
            double vv = v_after(m, V0, I0, tv);
            if (vv >= th) {
                c.hit = true;
                c.hi = tv;
                c.vhi = vv;
            }
        }
    }
    return c;
}

// Bracketed Newton-Raphson for the first time tau in (0, hi] with
// V(tau) = th (Appendix D.1), keeping [lo, hi] with V(lo) < th <= V(hi) and
// falling back to the midpoint whenever a step leaves the bracket (the
// clamp of D.1, i.e. a bisection step of D.2).  dV/dt comes from
// Eq. mem_dyn.  The start is the root of the chord from (0, V0) to
// (hi, V(hi)) instead of the paper's hi/2.  The iteration runs in float32
// (hardware exp) until its step is below float32 resolution, then float64
// steps finish it to float64 precision; the float64 bracket is kept
// throughout, so the float32 phase only supplies a starting point.
__device__ __forceinline__ double newton_root(const Model& m, double V0, double I0, double hi, double vhi,
                                              int* iters)
{
    double lo = 0.0;
    double t = (vhi > V0) ? hi * ((m.th - V0) / (vhi - V0)) : 0.5 * hi;
    if (!(t > 0.0 && t <= hi)) t = 0.5 * hi;
    int it = 0;
    {
        const float V0f = (float)V0, I0f = (float)I0, thf = (float)m.th, kf = (float)m.kappa;
        const float itm = (float)m.inv_tm, its = (float)m.inv_ts;
        float tf = (float)t, lof = 0.0f, hif = (float)hi;
        for (int k = 0; k < 24; ++k) {
            float em = __expf(-tf * itm), es = __expf(-tf * its);
            float v = V0f * em + I0f * kf * (em - es);
            if (v >= thf) hif = tf; else lof = tf;
            float dv = (I0f * es - v) * itm;
            float step = dv > 0.0f ? (v - thf) / dv : 0.0f;
            float tn = tf - step;
            if (!(tn > lof && tn < hif)) tn = 0.5f * (lof + hif);
            if (fabsf(tn - tf) <= 2e-7f * tf) { tf = tn; break; }
            tf = tn;
        }
        double tc = (double)tf;
        if (tc > 0.0 && tc < hi) t = tc;
    }
    for (; it < 96; ++it) {
        double em = exp(-t * m.inv_tm);
        double es = exp(-t * m.inv_ts);
        double v = V0 * em + I0 * m.kappa * (em - es);
        if (v >= m.th) hi = t; else lo = t;
        double d = (I0 * es - v) * m.inv_tm;
        double step = (d > 0.0) ? (v - m.th) / d : INFINITY;
        if (fabs(step) <= 2e-16 * t) { t -= step; break; }   // converged to the ulp
        double tn = t - step;
        if (!(tn > lo && tn < hi)) tn = 0.5 * (lo + hi);
        if (hi - lo <= 4e-16 * hi) { t = hi; break; }        // bracket collapsed
        t = tn;
    }
    if (iters) *iters = it;
    return t;
}

}  // namespace lif
