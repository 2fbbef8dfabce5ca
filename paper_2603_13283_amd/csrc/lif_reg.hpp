// lif_reg.hpp -- the per-interval pieces of the spike-count regularisers
// (Appendix E.1) shared by the plain and the delayed layer: the largest V of
// an interval (Eq. t_vmax) with its argmax, the per-interval record the
// gradient walks read, and its decoding.
#pragma once

#include "lif_common.hpp"

namespace lif {

// Largest V over [0, L] of the no-reset trajectory from (V0, I0): the start,
// the end (L finite) and the stationary point of Eq. t_vmax when it lies
// inside, with the decays e^{-u/tm}, e^{-u/ts} at its argmax and
// whether that is the interval's start or end (the first of equal values
// wins: the start, then the end, then the stationary point).
struct RegArg {
    double vmax, em, es;
    bool at_start, at_end;
};

__device__ __forceinline__ RegArg reg_vmax_arg(const Model& m, double V0, double I0, double L, double A, double Dd)
{
    RegArg r{V0, 1.0, 1.0, true, false};
    if (!isinf(L)) {
        const double V1 = V0 * A + m.kappa * I0 * (A - Dd);
        if (V1 > r.vmax) r = RegArg{V1, A, Dd, false, true};
    }
    // The logarithm and the decays of the stationary point in float32
    // arithmetic (relative errors near 2^-22; the records keep the decays in
    // float32 anyway), with e^{-u/ts} = (e^{-u/tm})^(p+1) when tau_m / tau_s
    // = p + 1; a ratio past the float32 range takes the float64 logarithm.
    const double a = V0 + m.kappa * I0;
    if (I0 > 0.0 && a > 0.0) {
        const double ratio = m.kappa * I0 * m.tm / (a * m.ts);
        if (ratio > 1.0) {
            const double u = (ratio < 1.0e38 ? (double)__logf((float)ratio) : log(ratio)) * m.c_tv;
            if (u > 0.0 && u < L) {
                const float emf = __expf((float)(-u * m.inv_tm));
                float esf;
                switch (m.p_int) {
                case 1: esf = emf * emf; break;
                case 2: esf = emf * emf * emf; break;
                case 3: { const float e2 = emf * emf; esf = e2 * e2; } break;
                case 4: { const float e2 = emf * emf; esf = e2 * e2 * emf; } break;
                default: esf = __expf((float)(-u * m.inv_ts)); break;
                }
                const double em = (double)emf, es = (double)esf;
                const double Vu = V0 * em + m.kappa * I0 * (em - es);
                if (Vu > r.vmax) r = RegArg{Vu, em, es, false, false};
            }
        }
    }
    return r;
}

// Per-interval record for the regularisers' gradient, interval j of a
// (sample, neuron), float2 {x, y} (the plain layer keeps them at
// rec[(b (E_max + 1) + j) N + n], the delayed one at
// rec[(b N + n)(E_max + 1) + j]).  An inactive interval (no hinge active)
// is {0, 0}.  For an active one the sign of x is the hinge (+ under-firing:
// silent with V_max < V_th; - over-firing: spiked with V_max > V_th) and |x|
// the argmax: kRecStartCode for the interval's start, kRecEndCode for its
// end (then y = the slope V' there when that point is an input time, else
// 0; the decays of an end are the interval's own), else e^{-u/tm} of a
// stationary point inside (or of the end t_end of the open interval), with
// y = e^{-u/ts}.
enum RecKind { kRecInside = 0, kRecStart = 1, kRecEnd = 2 };
constexpr float kRecStartCode = 2.0f, kRecEndCode = 3.0f;

__device__ __forceinline__ float2 make_record(float sgn, int kind, double em, double es, double slope)
{
    if (sgn == 0.0f) return make_float2(0.0f, 0.0f);
    if (kind == kRecStart) return make_float2(sgn * kRecStartCode, (float)slope);
    if (kind == kRecEnd) return make_float2(sgn * kRecEndCode, (float)slope);
    return make_float2(sgn * (float)em, (float)es);
}

// A record decoded with the interval's own decays (A, D): the multiplier mu
// of its pseudo-spike (dL/dV_max; 0 for an inactive record), the decays at
// its argmax, and its end-point slope terms: vs when the argmax is the start
// (the input event before the interval), ve when it is the end (the event
// that closes it), 0 otherwise.  Selects only, so that the walk over a group
// has no branches.
struct RecTerm {
    double mu, em, es, vs, ve;
};

__device__ __forceinline__ RecTerm rec_term(const float2& r, const double2& G, double A, double D)
{
    const float a = fabsf(r.x);
    const bool st = a == kRecStartCode, en = a == kRecEndCode;
    RecTerm t;
    t.mu = r.x > 0.0f ? G.x : (r.x < 0.0f ? G.y : 0.0);
    t.em = st ? 1.0 : (en ? A : (double)a);
    t.es = st ? 1.0 : (en ? D : (double)r.y);
    t.vs = st ? (double)r.y : 0.0;
    t.ve = en ? (double)r.y : 0.0;
    return t;
}

}  // namespace lif
