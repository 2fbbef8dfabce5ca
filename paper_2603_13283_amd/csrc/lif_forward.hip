// lif_forward.hip -- forward pass of the event-driven LIF layer on gfx950.
//
// Pipeline for one call (one sample = one event queue; N neurons share it):
//   k_decay      per (sample, event): the event's affine map M(dt) of
//                Eq. affine depends only on the gap to the previous event, so
//                its three entries (and a no-crossing bound factor) are
//                computed once per sample and shared by every neuron; per
//                segment of kSeg events also the composed map M(T_seg)
//                (the maps form a semigroup: M(a) M(b) = M(a + b)).
//   k_aggregate  per (sample, 64-neuron tile, segment): one wave walks the
//                segment's events from the zero state; lanes are neurons and
//                read their weight of each event from the event's W^T row
//                (one coalesced 256-byte row slice per event).  The result is
//                the b-part of the Combine of the segment's maps.
//   k_carry      per (sample, neuron): exclusive Combine scan over segments,
//                giving the no-reset state entering every segment.
//   k_check      per (sample, tile, segment): re-walk from the carried state
//                and test every inter-event interval with the paper's
//                interval rule (Sec. 3.2.2) behind a cheap exact upper bound.
//                Because resets only lower V, a segment whose no-reset
//                trajectory never reaches threshold cannot hold a spike, so
//                only flagged sub-blocks of kSub events are kept (with their
//                entering state and an upper bound of V over them).
//   k_resolve    per (sample, neuron): walks only its flagged sub-blocks in
//                time order.  Spikes found so far lower V by a known decaying
//                amount (the reset deficit), which both corrects the entering
//                state and certifies later sub-blocks without walking them.
//                A walked sub-block resolves spikes exactly: interval rule,
//                bracketed Newton (Appendix D.1), hard reset of V, re-test of
//                the same interval from the spike (Appendix E.2).
// The sequential baseline k_sequential (Appendix E.3) runs the same interval
// rule and root solve one event at a time per (sample, neuron).
#include "lif_common.hpp"
#include "lif_host.hpp"

namespace lif {

struct alignas(32) SubCarry {
    double V, I;    // no-reset state entering the sub-block
    double ub;      // upper bound of the no-reset V over the flagged intervals
    double pad;
};

// Workgroup index -> work index such that each of the 8 XCDs (which receive
// workgroups round-robin) processes a contiguous, sample-major range: the
// events and decays of a sample then stay in one XCD's L2.
__device__ __forceinline__ int xcd_remap(int wg, int total)
{
    int xcd = wg & 7, local = wg >> 3;
    int per = (total + 7) >> 3;
    int full = (total & 7) ? (total & 7) : 8;
    int base = xcd < full ? xcd * per : full * per + (xcd - full) * (per - 1);
    return base + local;
}

// ---------------------------------------------------------------------------
// k_decay
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_decay(const float* __restrict__ ev_t, const int32_t* __restrict__ ev_n,
                                               int B, int E_max, int S, Model m, Decay* __restrict__ dec,
                                               Decay* __restrict__ segm, int32_t* __restrict__ status)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx < LIF_STATUS_WORDS && status) status[idx] = 0;
    if (idx >= (size_t)B * (size_t)E_max) return;
    int b = (int)(idx / (size_t)E_max), k = (int)(idx % (size_t)E_max);
    int n = clamp_count(ev_n[b], E_max);
    if (k >= n) return;
    const float* t = ev_t + (size_t)b * E_max;
    double tk = (double)t[k];
    double tp = k > 0 ? (double)t[k - 1] : 0.0;
    double dt = tk - tp;
    Decay d;
    d.A = exp(-dt * m.inv_tm);
    d.D = exp(-dt * m.inv_ts);
    d.C = unit_kernel(m, dt, d.A);
    double gl = fmin(dt, m.t_peak);
    d.g = unit_kernel(m, gl, exp(-gl * m.inv_tm)) * (1.0 + 1e-12);
    dec[idx] = d;
    if (k % kSeg == 0) {
        int k1 = min(k + kSeg, n);
        double T = (double)t[k1 - 1] - tp;
        Decay s;
        s.A = exp(-T * m.inv_tm);
        s.D = exp(-T * m.inv_ts);
        s.C = unit_kernel(m, T, s.A);
        s.g = T;
        segm[(size_t)b * S + k / kSeg] = s;
    }
}

// Optional input validation (LIF_VALIDATE).
__global__ __launch_bounds__(256) void k_validate(const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src,
                                                  const int32_t* __restrict__ ev_n, int B, int E_max, int C_in,
                                                  int32_t* __restrict__ status)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (size_t)B * (size_t)E_max) return;
    int b = (int)(idx / (size_t)E_max), k = (int)(idx % (size_t)E_max);
    if (k == 0 && (ev_n[b] < 0 || ev_n[b] > E_max)) atomicOr(&status[LIF_ST_FLAGS], LIF_WARN_BAD_COUNT);
    if (k >= clamp_count(ev_n[b], E_max)) return;
    float t = ev_t[idx];
    int f = 0;
    if (!isfinite(t) || t < 0.0f) f |= LIF_WARN_NONFINITE;
    if (k > 0 && !(ev_t[idx - 1] <= t)) f |= LIF_WARN_UNSORTED;
    int s = ev_src[idx];
    if (s < 0 || s >= C_in) f |= LIF_WARN_BAD_SOURCE;
    if (f) atomicOr(&status[LIF_ST_FLAGS], f);
}

// ---------------------------------------------------------------------------
// Walk of one segment from a given state: V <- A V + C I, I <- D I + w.
// The event source and decay record are wave-uniform (scalar loads); the
// weight load is a coalesced W^T row slice.  Events are consumed in batches
// of kSub so the loads of a batch are in flight together.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void k_aggregate(const int32_t* __restrict__ ev_src, const int32_t* __restrict__ ev_n,
                                                  int E_max, const float* __restrict__ WT, int C_in, int N, int tiles, int S,
                                                  int total, const Decay* __restrict__ dec,
                                                  double2* __restrict__ agg)
{
    int lin = xcd_remap(blockIdx.x, total);
    int tile = lin % tiles;
    int rest = lin / tiles;
    int seg = rest % S;
    int b = rest / S;
    int nb = clamp_count(ev_n[b], E_max);
    int k0 = seg * kSeg;
    if (k0 >= nb) return;
    int k1 = min(k0 + kSeg, nb);
    int n = tile * kWave + (int)threadIdx.x;
    int nc = min(n, N - 1);
    const float* wcol = WT + nc;
    const int32_t* src = ev_src + (size_t)b * E_max;
    const Decay* d = dec + (size_t)b * E_max;
    double V = 0.0, I = 0.0;
    int k = k0;
    for (; k + kSub <= k1; k += kSub) {
        float w[kSub];
#pragma unroll
        for (int j = 0; j < kSub; ++j) w[j] = wcol[(size_t)clamp_src(src[k + j], C_in) * (size_t)N];
#pragma unroll
        for (int j = 0; j < kSub; ++j) {
            Decay e = d[k + j];
            double Vn = e.A * V + e.C * I;
            I = e.D * I + (double)w[j];
            V = Vn;
        }
    }
    for (; k < k1; ++k) {
        float w = wcol[(size_t)clamp_src(src[k], C_in) * (size_t)N];
        Decay e = d[k];
        double Vn = e.A * V + e.C * I;
        I = e.D * I + (double)w;
        V = Vn;
    }
    if (n < N) agg[((size_t)b * S + seg) * N + n] = make_double2(V, I);
}

// Exclusive scan over segments of the Combine of Eq. affine:
// s_in(j+1) = M(T_j) s_in(j) + b_j, with s_in(0) = (0, 0).
__global__ __launch_bounds__(256) void k_carry(const int32_t* __restrict__ ev_n, int B, int E_max, int N, int S,
                                               const Decay* __restrict__ segm, const double2* __restrict__ agg,
                                               double2* __restrict__ carry)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (size_t)B * (size_t)N) return;
    int b = (int)(idx / (size_t)N), n = (int)(idx % (size_t)N);
    int Sb = (clamp_count(ev_n[b], E_max) + kSeg - 1) / kSeg;
    double V = 0.0, I = 0.0;
    for (int j = 0; j < Sb; ++j) {
        size_t o = ((size_t)b * S + j) * N + n;
        carry[o] = make_double2(V, I);
        Decay M = segm[(size_t)b * S + j];
        double2 a = agg[o];
        double Vn = M.A * V + M.C * I + a.x;
        I = M.D * I + a.y;
        V = Vn;
    }
}

// Exact interval test of one no-reset sub-block walk, run only for lanes
// whose cheap bound fired somewhere in the sub-block.  Returns whether any
// interval of the sub-block satisfies the interval rule at th_lo and the
// largest bound value of such intervals.
__device__ __noinline__ bool subblock_exact(const Model& m, const float* __restrict__ tt,
                                            const int32_t* __restrict__ src, const Decay* __restrict__ d,
                                            const float* __restrict__ wcol, int C_in, int N, int kq0, int kq1, int nb,
                                            double V, double I, double* ub_out)
{
    bool cand = false;
    double ub = -INFINITY;
    for (int k = kq0; k < kq1; ++k) {
        Decay e = d[k];
        double u = fmax(V, 0.0) + fmax(I, 0.0) * e.g;
        double Vn = e.A * V + e.C * I;
        if (u >= m.th_lo) {
            double len = (double)tt[k] - (k > 0 ? (double)tt[k - 1] : 0.0);
            Crossing c = interval_rule(m, V, I, len, e.A, e.D, Vn, m.th_lo);
            if (c.hit) { cand = true; ub = fmax(ub, u); }
        }
        I = e.D * I + (double)wcol[(size_t)clamp_src(src[k], C_in) * (size_t)N];
        V = Vn;
    }
    if (kq1 == nb) {
        // Interval after the last event, up to t_end (default +inf).
        double len = m.t_end - (double)tt[nb - 1];
        if (len > 0.0) {
            double eA = isinf(len) ? 0.0 : exp(-len * m.inv_tm);
            double eD = isinf(len) ? 0.0 : exp(-len * m.inv_ts);
            double C = isinf(len) ? 0.0 : unit_kernel(m, len, eA);
            double gl = fmin(len, m.t_peak);
            double g = unit_kernel(m, gl, exp(-gl * m.inv_tm)) * (1.0 + 1e-12);
            double u = fmax(V, 0.0) + fmax(I, 0.0) * g;
            if (u >= m.th_lo) {
                Crossing c = interval_rule(m, V, I, len, eA, eD, V * eA + C * I, m.th_lo);
                if (c.hit) { cand = true; ub = fmax(ub, u); }
            }
        }
    }
    *ub_out = ub;
    return cand;
}

// Re-walk with the interval check.  Bound: V(t) = V0 e^{-t/tm} + I0 K(t)
// <= max(V0, 0) + max(I0, 0) K(min(dt, t_peak)) since 0 <= K <= that value
// on [0, dt].  The hot loop only records whether the bound reached th_lo in
// a sub-block (one compare per event); such sub-blocks, rare except right
// around spikes, are walked again with the exact interval rule.
__global__ __launch_bounds__(64) void k_check(const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src,
                                              const int32_t* __restrict__ ev_n, int E_max,
                                              const float* __restrict__ WT, int C_in, int N, int tiles, int S,
                                              int total, Model m, const Decay* __restrict__ dec,
                                              const double2* __restrict__ carry, uint32_t* __restrict__ mask,
                                              SubCarry* __restrict__ subc, int32_t* __restrict__ status)
{
    int lin = xcd_remap(blockIdx.x, total);
    int tile = lin % tiles;
    int rest = lin / tiles;
    int seg = rest % S;
    int b = rest / S;
    int nb = clamp_count(ev_n[b], E_max);
    int k0 = seg * kSeg;
    if (k0 >= nb) return;
    int k1 = min(k0 + kSeg, nb);
    int n = tile * kWave + (int)threadIdx.x;
    int nc = min(n, N - 1);
    const float* wcol = WT + nc;
    const float* tt = ev_t + (size_t)b * E_max;
    const int32_t* src = ev_src + (size_t)b * E_max;
    const Decay* d = dec + (size_t)b * E_max;
    size_t row = ((size_t)b * S + seg) * N;
    double2 c0 = carry[row + nc];
    double V = c0.x, I = c0.y;
    uint32_t msk = 0;
    int ncand = 0;
    for (int q = 0; q < kSubPerSeg; ++q) {
        int kq0 = k0 + q * kSub;
        if (kq0 >= k1) break;
        int kq1 = min(kq0 + kSub, k1);
        double Vin = V, Iin = I;
        bool surv = kq1 == nb;           // the open last interval is always tested exactly
        if (kq1 - kq0 == kSub) {
            float w[kSub];
#pragma unroll
            for (int j = 0; j < kSub; ++j) w[j] = wcol[(size_t)clamp_src(src[kq0 + j], C_in) * (size_t)N];
#pragma unroll
            for (int j = 0; j < kSub; ++j) {
                Decay e = d[kq0 + j];
                surv |= fmax(V, 0.0) + fmax(I, 0.0) * e.g >= m.th_lo;
                double Vn = e.A * V + e.C * I;
                I = e.D * I + (double)w[j];
                V = Vn;
            }
        } else {
            for (int k = kq0; k < kq1; ++k) {
                float w = wcol[(size_t)clamp_src(src[k], C_in) * (size_t)N];
                Decay e = d[k];
                surv |= fmax(V, 0.0) + fmax(I, 0.0) * e.g >= m.th_lo;
                double Vn = e.A * V + e.C * I;
                I = e.D * I + (double)w;
                V = Vn;
            }
        }
        if (surv && n < N) {
            double ub;
            if (subblock_exact(m, tt, src, d, wcol, C_in, N, kq0, kq1, nb, Vin, Iin, &ub)) {
                SubCarry sc;
                sc.V = Vin; sc.I = Iin; sc.ub = ub; sc.pad = 0.0;
                subc[row * kSubPerSeg + (size_t)q * N + n] = sc;
                msk |= 1u << q;
                ++ncand;
            }
        }
    }
    if (n < N) {
        mask[row + n] = msk;
        if (ncand) atomicAdd(&status[LIF_ST_CAND_BLOCKS], ncand);
    }
}

// ---------------------------------------------------------------------------
// Exact advance of one neuron across [t_cur, t_hi]: every spike inside is
// solved and followed by a hard reset and a re-test of the rest of the same
// interval.  `tab` holds the decays of the whole gap and is used while no
// spike has split the interval.  Returns false once the neuron is capped.
// ---------------------------------------------------------------------------
struct Sink {
    float* st;      // this neuron's s_max time slots
    float* si;      // this neuron's s_max current slots, may be null
    int ns;         // spikes so far
    int roots;      // root solves
    double dref;    // reset deficit at tref (sum of (th - vr) e^{-(t - t_s)/tm})
    double tref;
};

__device__ bool advance_interval(const Model& m, double& V, double& I, double& t_cur, double t_hi,
                                 const Decay* tab, Sink& sk)
{
    bool fresh = tab != nullptr;
    for (;;) {
        double len = t_hi - t_cur;
        if (!(len > 0.0)) return true;
        double eA, eD, C, g;
        if (fresh) {
            eA = tab->A; eD = tab->D; C = tab->C; g = tab->g;
        } else if (isinf(len)) {
            eA = 0.0; eD = 0.0; C = 0.0;
            g = unit_kernel(m, m.t_peak, exp(-m.t_peak * m.inv_tm)) * (1.0 + 1e-12);
        } else {
            eA = exp(-len * m.inv_tm);
            eD = exp(-len * m.inv_ts);
            C = unit_kernel(m, len, eA);
            double gl = fmin(len, m.t_peak);
            g = unit_kernel(m, gl, exp(-gl * m.inv_tm)) * (1.0 + 1e-12);
        }
        double vend = V * eA + C * I;
        double u = fmax(V, 0.0) + fmax(I, 0.0) * g;
        if (u >= m.th_lo) {
            Crossing c = interval_rule(m, V, I, len, eA, eD, vend, m.th);
            if (c.hit) {
                int it = 0;
                double tau = newton_root(m, V, I, c.hi, &it);
                double Istar = I * exp(-tau * m.inv_ts);
                double tsp = t_cur + tau;
                sk.st[sk.ns] = (float)tsp;
                if (sk.si) sk.si[sk.ns] = (float)Istar;
                sk.ns++;
                sk.roots++;
                sk.dref = sk.dref * exp(-(tsp - sk.tref) * m.inv_tm) + (m.th - m.vr);
                sk.tref = tsp;
                V = m.vr;
                I = Istar;
                t_cur = tsp;
                fresh = false;
                if (sk.ns >= m.s_max) return false;
                continue;
            }
        }
        V = vend;
        I = I * eD;
        t_cur = t_hi;
        return true;
    }
}

__device__ __forceinline__ void finish_neuron(const Model& m, Sink& sk, int32_t* out_n_slot, bool capped,
                                              int32_t* status)
{
    *out_n_slot = sk.ns;
    for (int s = sk.ns; s < m.s_max; ++s) {
        sk.st[s] = INFINITY;
        if (sk.si) sk.si[s] = 0.0f;
    }
    if (capped) {
        atomicAdd(&status[LIF_ST_CAPPED], 1);
        atomicOr(&status[LIF_ST_FLAGS], LIF_WARN_SPIKE_CAP);
    }
    if (sk.ns) atomicAdd(&status[LIF_ST_SPIKES], sk.ns);
    if (sk.roots) atomicAdd(&status[LIF_ST_ROOT_SOLVES], sk.roots);
}

__global__ __launch_bounds__(256) void k_resolve(const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src,
                                                 const int32_t* __restrict__ ev_n, int B, int E_max,
                                                 const float* __restrict__ WT, int C_in, int N, int S, Model m,
                                                 const Decay* __restrict__ dec, const uint32_t* __restrict__ mask,
                                                 const SubCarry* __restrict__ subc, float* __restrict__ out_t,
                                                 int32_t* __restrict__ out_n, float* __restrict__ out_i,
                                                 int32_t* __restrict__ status)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (size_t)B * (size_t)N) return;
    int b = (int)(idx / (size_t)N), n = (int)(idx % (size_t)N);
    int nb = clamp_count(ev_n[b], E_max);
    if (n == 0) atomicAdd(&status[LIF_ST_EVENTS], nb);
    const float* tt = ev_t + (size_t)b * E_max;
    const int32_t* src = ev_src + (size_t)b * E_max;
    const Decay* d = dec + (size_t)b * E_max;
    Sink sk;
    sk.st = out_t + idx * (size_t)m.s_max;
    sk.si = out_i ? out_i + idx * (size_t)m.s_max : nullptr;
    sk.ns = 0; sk.roots = 0; sk.dref = 0.0; sk.tref = 0.0;
    bool capped = false;
    int walked = 0;
    int Sb = (nb + kSeg - 1) / kSeg;
    for (int seg = 0; seg < Sb && !capped; ++seg) {
        size_t row = ((size_t)b * S + seg) * N;
        uint32_t msk = mask[row + n];
        while (msk && !capped) {
            int q = __builtin_ctz(msk);
            msk &= msk - 1;
            SubCarry sc = subc[row * kSubPerSeg + (size_t)q * N + n];
            int kq0 = seg * kSeg + q * kSub;
            int kq1 = min(kq0 + kSub, nb);
            bool last = kq1 == nb;
            double t_in = kq0 > 0 ? (double)tt[kq0 - 1] : 0.0;
            // End of the sub-block's last interval (the open interval after the
            // final event ends at t_end, or is empty if t_end is earlier).
            double t_out = last ? fmax(m.t_end, (double)tt[kq1 - 1]) : (double)tt[kq1 - 1];
            double def_in = 0.0;
            if (sk.ns > 0) {
                double def_out = isinf(t_out) ? 0.0 : sk.dref * exp(-(t_out - sk.tref) * m.inv_tm);
                if (sc.ub - def_out < m.th_lo) continue;    // certified by the deficit
                def_in = sk.dref * exp(-(t_in - sk.tref) * m.inv_tm);
            }
            ++walked;
            double V = sc.V - def_in, I = sc.I, t_cur = t_in;
            for (int k = kq0; k < kq1; ++k) {
                if (!advance_interval(m, V, I, t_cur, (double)tt[k], &d[k], sk)) { capped = true; break; }
                I += (double)WT[(size_t)clamp_src(src[k], C_in) * (size_t)N + n];
            }
            if (!capped && last) {
                if (!advance_interval(m, V, I, t_cur, m.t_end, nullptr, sk)) capped = true;
            }
        }
    }
    if (walked) atomicAdd(&status[LIF_ST_WALKED_BLOCKS], walked);
    finish_neuron(m, sk, out_n + idx, capped, status);
}

// Sequential baseline: one thread per (sample, neuron), every event in order.
__global__ __launch_bounds__(64) void k_sequential(const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src,
                                                   const int32_t* __restrict__ ev_n, int B, int E_max,
                                                   const float* __restrict__ WT, int C_in, int N, Model m,
                                                   const Decay* __restrict__ dec, float* __restrict__ out_t,
                                                   int32_t* __restrict__ out_n, float* __restrict__ out_i,
                                                   int32_t* __restrict__ status)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (size_t)B * (size_t)N) return;
    int b = (int)(idx / (size_t)N), n = (int)(idx % (size_t)N);
    int nb = clamp_count(ev_n[b], E_max);
    if (n == 0) atomicAdd(&status[LIF_ST_EVENTS], nb);
    const float* tt = ev_t + (size_t)b * E_max;
    const int32_t* src = ev_src + (size_t)b * E_max;
    const Decay* d = dec + (size_t)b * E_max;
    Sink sk;
    sk.st = out_t + idx * (size_t)m.s_max;
    sk.si = out_i ? out_i + idx * (size_t)m.s_max : nullptr;
    sk.ns = 0; sk.roots = 0; sk.dref = 0.0; sk.tref = 0.0;
    double V = 0.0, I = 0.0, t_cur = 0.0;
    bool capped = false;
    for (int k = 0; k < nb; ++k) {
        if (!advance_interval(m, V, I, t_cur, (double)tt[k], &d[k], sk)) { capped = true; break; }
        I += (double)WT[(size_t)clamp_src(src[k], C_in) * (size_t)N + n];
    }
    if (!capped && !advance_interval(m, V, I, t_cur, m.t_end, nullptr, sk)) capped = true;
    finish_neuron(m, sk, out_n + idx, capped, status);
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
FwdLayout fwd_layout(int B, int E_max, int N)
{
    FwdLayout L{};
    L.S = (E_max + kSeg - 1) / kSeg;
    size_t off = 0;
    auto take = [&](size_t bytes) { size_t o = off; off += (bytes + 255) & ~(size_t)255; return o; };
    L.dec = take((size_t)B * E_max * sizeof(Decay));
    L.segm = take((size_t)B * L.S * sizeof(Decay));
    L.agg = take((size_t)B * L.S * N * sizeof(double2));
    L.carry = take((size_t)B * L.S * N * sizeof(double2));
    L.mask = take((size_t)B * L.S * N * sizeof(uint32_t));
    L.subc = take((size_t)B * L.S * kSubPerSeg * N * sizeof(SubCarry));
    L.total = off + 256;
    return L;
}

int forward_impl(bool sequential, const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                 const float* WT, int C_in, int N, const lif_params* p, float* out_t, int32_t* out_n,
                 float* out_i, int32_t* status, void* ws, size_t ws_bytes, hipStream_t stream)
{
    int rc = validate_forward_args(ev_t, ev_src, ev_n, B, E_max, WT, C_in, N, p, out_t, out_n, status, ws);
    if (rc) return rc;
    FwdLayout L = fwd_layout(B, E_max, N);
    if (ws_bytes < L.total) return LIF_ERR_WORKSPACE;
    Model m = make_model(*p);
    char* base = (char*)(((uintptr_t)ws + 255) & ~(uintptr_t)255);
    Decay* dec = (Decay*)(base + L.dec);
    Decay* segm = (Decay*)(base + L.segm);
    double2* agg = (double2*)(base + L.agg);
    double2* carry = (double2*)(base + L.carry);
    uint32_t* mask = (uint32_t*)(base + L.mask);
    SubCarry* subc = (SubCarry*)(base + L.subc);

    size_t nev = (size_t)B * E_max;
    size_t dec_threads = nev > LIF_STATUS_WORDS ? nev : LIF_STATUS_WORDS;
    TIMED_LAUNCH("decay", k_decay, dim3((unsigned)((dec_threads + 255) / 256)), dim3(256), 0, stream,
                 ev_t, ev_n, B, E_max, L.S, m, dec, segm, status);
    if ((p->flags & LIF_VALIDATE) && nev)
        TIMED_LAUNCH("validate", k_validate, dim3((unsigned)((nev + 255) / 256)), dim3(256), 0, stream,
                     ev_t, ev_src, ev_n, B, E_max, C_in, status);
    size_t nn = (size_t)B * N;
    if (sequential) {
        TIMED_LAUNCH("sequential", k_sequential, dim3((unsigned)((nn + 63) / 64)), dim3(64), 0, stream,
                     ev_t, ev_src, ev_n, B, E_max, WT, C_in, N, m, dec, out_t, out_n, out_i, status);
        return check_launch();
    }
    int tiles = (N + kWave - 1) / kWave;
    size_t total = (size_t)B * L.S * tiles;
    if (total > 0x7fffffff) return LIF_ERR_SIZE;
    if (total) {
        TIMED_LAUNCH("aggregate", k_aggregate, dim3((unsigned)total), dim3(kWave), 0, stream,
                     ev_src, ev_n, E_max, WT, C_in, N, tiles, L.S, (int)total, dec, agg);
        TIMED_LAUNCH("carry", k_carry, dim3((unsigned)((nn + 255) / 256)), dim3(256), 0, stream,
                     ev_n, B, E_max, N, L.S, segm, agg, carry);
        TIMED_LAUNCH("check", k_check, dim3((unsigned)total), dim3(kWave), 0, stream,
                     ev_t, ev_src, ev_n, E_max, WT, C_in, N, tiles, L.S, (int)total, m, dec, carry, mask, subc, status);
    }
    TIMED_LAUNCH("resolve", k_resolve, dim3((unsigned)((nn + 255) / 256)), dim3(256), 0, stream,
                 ev_t, ev_src, ev_n, B, E_max, WT, C_in, N, L.S, m, dec, mask, subc, out_t, out_n, out_i, status);
    return check_launch();
}

}  // namespace lif

extern "C" size_t lif_layer_forward_workspace_size(int B, int E_max, int C_in, int N_out, const lif_params* p)
{
    (void)C_in; (void)p;
    if (B < 0 || E_max < 0 || N_out < 1) return 0;
    return lif::fwd_layout(B, E_max, N_out).total;
}

extern "C" int lif_layer_forward(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                                 const float* WT, int C_in, int N_out, const lif_params* p, float* out_t,
                                 int32_t* out_n, float* out_i, int32_t* status, void* ws, size_t ws_bytes,
                                 lif_stream_t stream)
{
    return lif::forward_impl(false, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, p, out_t, out_n, out_i, status,
                             ws, ws_bytes, (hipStream_t)stream);
}

extern "C" int lif_layer_forward_sequential(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B,
                                            int E_max, const float* WT, int C_in, int N_out, const lif_params* p,
                                            float* out_t, int32_t* out_n, float* out_i, int32_t* status, void* ws,
                                            size_t ws_bytes, lif_stream_t stream)
{
    return lif::forward_impl(true, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, p, out_t, out_n, out_i, status,
                             ws, ws_bytes, (hipStream_t)stream);
}
