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
constexpr int kSeg = 64;        // events per scan segment (one wave walks it)
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
    double th_lo;      // survival threshold of the no-crossing screen (slightly below th)
    double thk_lo;     // th_lo / kappa: the same threshold in the eigen-coordinates of the walks
    double inv_ktm;    // 1 / (kappa tau_m)
    double inv_th;     // 1 / th
    double th_1k;      // th (1 + kappa)
    double ts_tm;      // tau_s / tau_m
    double dth;        // th - vr: the drop of V at a reset
    double reg;        // backward floor on dV/dt
    float f_th, f_inv_tm;   // float32 copies for screening
    int p_int;         // p when tau_m / tau_s = p + 1 exactly for an integer 1 <= p <= 4, else 0
    int s_max;
    uint32_t flags;
};

// Per-event decay record, shared by every neuron of a sample (the matrix
// M(dt) of Eq. affine depends only on the gap dt to the previous event):
//   A = e^{-dt/tm}, D = e^{-dt/ts}, C = kappa (e^{-dt/tm} - e^{-dt/ts}),
//   lk = dt / (kappa tm): the slope factor of the no-crossing screen.
// Padding entries past a sample's last event hold the identity map
// (A = D = 1, C = lk = 0).
struct alignas(32) Decay {
    double A, D, C, lk;
};

// Eigen-coordinates of the event map.  M(dt) = [[A, C], [0, D]] has the
// eigenvalues A and D; with U = V / kappa + I and J = I the state decays as
// two independent exponentials, U -> A U and J -> D J, an input of weight w
// adds w to both (it raises I and leaves V unchanged), and
// V = kappa (U - J), I = J.  This is Eq. mem_pot (V = (V0 + kappa I0)
// e^{-t/tm} - kappa I0 e^{-t/ts}) with both terms divided by kappa.
__device__ __forceinline__ double v_of(const Model& m, double U, double J) { return m.kappa * (U - J); }
__device__ __forceinline__ double u_of(const Model& m, double V, double I) { return V / m.kappa + I; }

// No-crossing screen of one interval of length L = lk kappa tm that starts
// in the no-reset state (U, J): the interval can reach the threshold only if
//   (U - J) + max(J - th, 0) lk >= th_lo / kappa,
// i.e. V0 + max(I0 - th, 0) L / tm >= th_lo.  Proof: with
// h(u) = (V_lin(u) - th) e^{u/tm}, h'(u) = (I0 e^{-u (1/ts - 1/tm)} - th
// e^{u/tm}) / tm; for I0 > th, h is concave and lies below its tangent at 0,
// h(0) + h'(0) u = V0 - th + (I0 - th) u / tm; for I0 <= th, h is
// decreasing and its maximum is h(0) = V0 - th.  Resets only lower V
// (Sec. 3.1: the reset subtracts a positive decaying term), so an interval
// that fails the screen for the no-reset state holds no spike.
__device__ __forceinline__ double screen_value(const Model& m, double U, double J, double lk)
{
    return fma(fmax(J - m.th, 0.0), lk, U - J);
}

// Source channel of an event, clamped into [0, C_in) so that a malformed
// queue can never address outside W (LIF_VALIDATE reports such events).
__device__ __forceinline__ int clamp_src(int s, int C_in) { return min(max(s, 0), C_in - 1); }

// Event count of a sample, clamped into [0, E_max].
__device__ __forceinline__ int clamp_count(int n, int E_max) { return min(max(n, 0), E_max); }

// Adjoints of one neuron's spikes (Appendix D.3, Eq. ift_vjp, chained
// through the hard resets), last spike first:
//   lambda_s = g_s - ((V_th - V_reset)/tm) sum_{s'' > s} mu_s'' e^{-(t_s'' - t_s)/tm}
//   mu_s     = -lambda_s / max(dV/dt(t_s), reg),  dV/dt(t_s) = (I_s - V_th)/tm
// (mo[s] = mu_s).  Returns sum_s |mu_s|, which bounds the neuron's adjoint
// sums P^m and P^s.
__device__ inline double spike_adjoints(const Model& m, int ns, const float* __restrict__ ts,
                                        const float* __restrict__ is, const float* __restrict__ g,
                                        double* __restrict__ mo)
{
    const double jump = (m.th - m.vr) * m.inv_tm;
    double Q = 0.0, mu_next = 0.0, asum = 0.0;
    for (int s = ns - 1; s >= 0; --s) {
        if (s + 1 < ns) Q = (Q + mu_next) * exp(-((double)ts[s + 1] - (double)ts[s]) * m.inv_tm);
        const double lam = (double)g[s] - jump * Q;
        const double vp = fmax(((double)is[s] - m.th) * m.inv_tm, m.reg);
        const double mu_s = vp > 0.0 ? -lam / vp : 0.0;
        mo[s] = mu_s;
        mu_next = mu_s;
        asum += fabs(mu_s);
    }
    return asum;
}

// Unit kernel K(u) = kappa (e^{-u/tm} - e^{-u/ts}) written with expm1 so that
// tiny gaps do not cancel.
__device__ __forceinline__ double unit_kernel(const Model& m, double u, double eA)
{
    return -m.kappa * eA * expm1(-u * m.a_rate);
}

// Interval test in deficit form.  Every spike at t_s lowers V afterwards by
// (th - vr) e^{-(t - t_s)/tm} (hard reset of a linear system, Sec. 3.1 and
// Eq. mem_pot), so on an interval that starts at the no-reset state
// (V0, I0) with the spikes so far amounting to a deficit D at its start, the
// true potential is V_lin(u) - D e^{-u/tm}, u in [0, L].  It reaches th
// inside (0, L] iff D <= max h over (0, L] with
//   h(u) = (V_lin(u) - th) e^{u/tm}
//        = V0 - th e^{u/tm} + kappa I0 (1 - e^{-u r}),   r = 1/ts - 1/tm.
// h'(u) = (I0 e^{-u r} - th e^{u/tm}) / tm: for th > 0 the only stationary
// point is u* = ts ln(I0/th), a maximum, where h(u*) =
// V0 + kappa I0 - th (1 + kappa) (I0/th)^{ts/tm}; it lies inside (0, L) iff
// I0 > th and I0 e^{-L/ts} < th.  Otherwise h is monotone on the interval
// and the test is the end value, D e^{-L/tm} <= V_lin(L) - th.  This is the
// interval rule of Sec. 3.2.2 (t_Vmax of Eq. t_vmax, V at the maximum or at
// the end) applied to V_lin - D e^{-u/tm}, with the maximum taken of h so
// that the deficit enters as a single multiply: the test does not change as
// D grows, and a spike in the interval re-tests the rest of it (the maximum
// over (u_s, L] is the same, since u_s <= u*).
struct IntervalMax {
    double g;     // crossing iff D * a <= g
    double a;     // 1 (interior maximum) or e^{-L/tm} (end value)
    double hi;    // right end of the root bracket: u* or L
    double Fhi;   // h(hi); F(hi) = h(hi) - D starts the root solve
};

__device__ __forceinline__ IntervalMax interval_max(const Model& m, double V0, double I0, double V1, double L,
                                                    double A, double D)
{
#pragma clang fp contract(off)      // the same IEEE operations wherever it is inlined
    IntervalMax r;
    if (I0 > m.th && I0 * D < m.th) {
        double lr = log(I0 * m.inv_th);
        r.g = V0 + m.kappa * I0 - m.th_1k * exp(m.ts_tm * lr);
        r.a = 1.0;
        r.hi = m.ts * lr;
        r.Fhi = r.g;
    } else {
        r.g = V1 - m.th;
        r.a = A;
        r.hi = L;
        r.Fhi = A > 0.0 ? r.g / A : -INFINITY;
    }
    return r;
}

// e^x for |x| <= 4e-3 by its Taylor series to x^6 (relative error < 1e-17).
__device__ __forceinline__ double exp_small(double x)
{
    return 1.0 + x * (1.0 + x * (0.5 + x * (1.0 / 6.0 + x * (1.0 / 24.0 + x * (1.0 / 120.0 + x * (1.0 / 720.0))))));
}

// 1/x from the hardware reciprocal refined by one Newton step (error of a
// few ulp; used where a quotient only has to be accurate to ~1e-15).
__device__ __forceinline__ double rcp_refined(double x)
{
    double r = __builtin_amdgcn_rcp(x);
    return r * (2.0 - x * r);
}

// One step of the bracketed Newton iteration of root_h, written without
// branches except for the rare exact re-evaluation of the exponentials.
__device__ __forceinline__ void newton_step(const Model& m, double c0, double kI, double dF1, double dF2, double rmax,
                                            double& u, double& lo, double& hi, double& E1, double& E2, double& d)
{
    const double F = c0 - m.th * E1 - kI * E2;
    const bool pos = F >= 0.0;
    hi = pos ? u : hi;
    lo = pos ? lo : u;
    const double dF = dF1 * E2 - dF2 * E1;
    double un = u - F * rcp_refined(dF);
    un = (dF > 0.0 && un > lo && un < hi) ? un : 0.5 * (lo + hi);
    un = (F == 0.0 || !(hi - lo > 4e-16 * hi)) ? u : un;     // exact root, or bracket collapsed onto u
    d = un - u;
    if (fabs(d) * rmax <= 4e-3) {
        E1 *= exp_small(d * m.inv_tm);
        E2 *= exp_small(-d * m.a_rate);
    } else {
        E1 = exp(un * m.inv_tm);
        E2 = exp(-un * m.a_rate);
    }
    u = un;
}

// Spike time inside a crossing interval (Appendix D.1, bracketed
// Newton-Raphson): the smallest u in (lo, hi] with F(u) = h(u) - D = 0,
//   F(u) = c0 - th e^{u/tm} - kI e^{-u r},  c0 = V0 - D + kappa I0, kI = kappa I0,
// given F(lo) = Flo < 0 <= F(hi) = Fhi.  F is concave wherever it can cross
// (I0 > 0), so it increases through its first root.  The iteration keeps
// [lo, hi] with F(lo) < 0 <= F(hi) and takes the midpoint whenever a Newton
// step leaves it (the clamp of D.1).  Instead of the paper's midpoint start:
//   * a float32 Newton phase (hardware exponentials) from the root of the
//     chord from (lo, Flo) to (hi, Fhi) brings u to float32 accuracy;
//   * float64 Newton steps then run from there with the two exponentials
//     evaluated exactly once and carried along by the factor e^{step}
//     (Taylor series) while steps are small.  The iteration stops when a
//     step is below 1e-9 ts, or below 1e-7 ts and at most 1/100 of the step
//     before it (quadratic convergence: the error left is then far below
//     float64 resolution of the spike time), or the bracket collapses.
// On return *E1 = e^{u/tm} and *E2 = e^{-u r} at the returned u.
__device__ __forceinline__ double root_h(const Model& m, double c0, double kI, double lo, double Flo, double hi,
                                         double Fhi, double* E1o, double* E2o, int* iters)
{
    double u = (Fhi > Flo && Fhi < INFINITY) ? lo + (hi - lo) * (-Flo * rcp_refined(Fhi - Flo)) : 0.5 * (lo + hi);
    if (!(u > lo && u <= hi)) u = 0.5 * (lo + hi);
    {
        // float32 phase (a start value only: the float64 phase below is
        // bracketed and does not rely on it)
        const float c0f = (float)c0, kIf = (float)kI, thf = (float)m.th, itm = (float)m.inv_tm,
                    ar = (float)m.a_rate;
        float lf = (float)lo, hf = (float)hi, uf = (float)u;
#pragma unroll 1
        for (int i = 0; i < 3; ++i) {
            const float e1 = __expf(uf * itm), e2 = __expf(-uf * ar);
            const float F = c0f - thf * e1 - kIf * e2;
            const float dF = kIf * ar * e2 - thf * itm * e1;
            if (F >= 0.0f) hf = uf; else lf = uf;
            float un = uf - F / dF;
            if (!(dF > 0.0f && un > lf && un < hf)) un = 0.5f * (lf + hf);
            uf = un;
        }
        const double ud = (double)uf;
        if (ud > lo && ud <= hi) u = ud;
    }
    double E1 = exp(u * m.inv_tm), E2 = exp(-u * m.a_rate);
    const double tol = 1e-9 * m.ts, tol_q = 1e-7 * m.ts;
    const double dF1 = kI * m.a_rate, dF2 = m.th * m.inv_tm;
    const double rmax = fmax(m.inv_tm, m.a_rate);
    double d = 0.0, dprev = INFINITY;
    int it = 0;
#pragma unroll 1
    while (it < 96) {
        newton_step(m, c0, kI, dF1, dF2, rmax, u, lo, hi, E1, E2, d);
        ++it;
        const double ad = fabs(d);
        if (ad <= tol || (ad <= tol_q && ad <= 0.01 * dprev)) break;
        dprev = ad;
    }
    *E1o = E1;
    *E2o = E2;
    if (iters) *iters += it;
    return u;
}

// Spike time when tau_m / tau_s = p + 1 for an integer 1 <= p <= 4 (the
// paper's 20 ms / 5 ms gives p = 3).  With y = e^{-u/tm} the two
// exponentials of F become powers of y: e^{u/tm} = 1/y and e^{-u r} = y^p, so
//   P(y) = -y F(u) = kI y^{p+1} - c0 y + th
// is a polynomial.  A crossing interval has kI > 0, where P is convex in
// y > 0; its first root in u is the largest root in y, and P(ylo) =
// -ylo F(lo) > 0 at the bracket end ylo = e^{-lo/tm}, so Newton steps from
// ylo decrease monotonically onto that root.  Four float32 steps (hardware
// reciprocal) bring y near float32 resolution, float64 steps finish; no
// exponential or logarithm is evaluated.  Returns false when an iteration
// leaves this pattern (non-increasing P, no convergence), which exact
// arithmetic excludes; the caller then takes root_h.
template <int P, typename T>
__device__ __forceinline__ T ipow(T y)
{
    if constexpr (P == 0) {
        return T(1);
    } else {
        T r = y;
#pragma unroll
        for (int i = 1; i < P; ++i) r *= y;
        return r;
    }
}

template <int P>
__device__ __forceinline__ bool root_poly(const Model& m, double c0, double kI, double ylo, double& y_out)
{
    {
        const float c0f = (float)c0, kIf = (float)kI, thf = (float)m.th, kp1f = (float)(P + 1) * kIf;
        float y = (float)ylo;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float yp = ipow<P>(y);
            const float Pv = fmaf(kIf * yp, y, fmaf(-c0f, y, thf));
            const float dP = fmaf(kp1f, yp, -c0f);
            const float yn = y - Pv * __builtin_amdgcn_rcpf(dP);
            y = (dP > 0.0f && yn > 0.0f && yn < y) ? yn : y;
        }
        // the float32 iterate may sit a rounding step left of the root;
        // the float64 steps below converge from either side
        y_out = (double)y;
    }
    const double kp1 = (double)(P + 1) * kI;
    const double half_d2 = 0.5 * (double)(P * (P + 1)) * kI;   // P''(y) / 2 = half_d2 y^(P-1)
    double y = y_out;
#pragma unroll 1
    for (int it = 0; it < 64; ++it) {
        const double ym = ipow<P - 1>(y);
        const double yp = ym * y;
        const double Pv = fma(kI * yp, y, fma(-c0, y, m.th));
        const double dP = fma(kp1, yp, -c0);
        if (!(dP > 0.0)) return false;
        const double rdP = rcp_refined(dP);
        const double step = Pv * rdP;
        y -= step;
        if (!(y > 0.0 && y <= ylo)) return false;
        // converged: the error left after a Newton step of size s is about
        // P'' s^2 / (2 P') (Taylor's theorem), trusted once the step is
        // small; it must lie below 2^-40 y (spike times and reset deficits
        // then carry errors far below the float32 outputs' resolution)
        const double as = fabs(step);
        if (as <= 0x1p-48 * y || (as <= 0x1p-20 * y && half_d2 * ym * (as * as) * rdP <= 0x1p-40 * y)) {
            y_out = y;
            return true;
        }
    }
    return false;
}

// Spike inside a crossing interval (F(lo) = Flo < 0 <= F(hi) = Fhi, ylo =
// e^{-lo/tm}): y = e^{-u/tm} at the spike time u, E1 = e^{u/tm},
// E2 = e^{-u r}.  The spike time itself is u = -tm ln y.
struct SpikeY {
    double y, E1, E2;
};

__device__ __forceinline__ SpikeY solve_spike_y(const Model& m, double c0, double kI, double lo, double ylo, double Flo,
                                                double hi, double Fhi)
{
    SpikeY r;
    double y = 0.0;
    bool ok = false;
    switch (m.p_int) {
    case 1: ok = root_poly<1>(m, c0, kI, ylo, y); if (ok) r.E2 = y; break;
    case 2: ok = root_poly<2>(m, c0, kI, ylo, y); if (ok) r.E2 = ipow<2>(y); break;
    case 3: ok = root_poly<3>(m, c0, kI, ylo, y); if (ok) r.E2 = ipow<3>(y); break;
    case 4: ok = root_poly<4>(m, c0, kI, ylo, y); if (ok) r.E2 = ipow<4>(y); break;
    default: break;
    }
    if (ok) {
        r.y = y;
        r.E1 = rcp_refined(y);
    } else {
        root_h(m, c0, kI, lo, Flo, hi, Fhi, &r.E1, &r.E2, nullptr);
        r.y = rcp_refined(r.E1);
    }
    return r;
}

}  // namespace lif
