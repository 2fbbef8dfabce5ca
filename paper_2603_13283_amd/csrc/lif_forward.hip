// lif_forward.hip -- forward pass of the event-driven LIF layer on gfx950.
//
// Pipeline for one call (a sample is one sorted event queue, shared by the
// N neurons of the layer):
//   k_aggregate  per (sample, segment, tile of 64 NPL neurons): the affine
//                map M(dt) of Eq. affine depends only on the gap to the
//                previous event, so the segment's maps are computed once per
//                sample (the first tile's wave stores them, and the composed
//                map of the segment: the maps form a semigroup,
//                M(a) M(b) = M(a + b)) and shared by every neuron.  One wave walks
//                the segment from the zero state in the eigen-coordinates
//                (U, J) of the maps (two FMAs per neuron-event, the decays as
//                scalar operands).  Lane l holds NPL adjacent neurons and
//                reads their weights of an event with one vector load from
//                the event's W^T row.  The result is the b-part of the
//                Combine of the segment's maps.
//   k_carry      per (sample, 64 neurons): exclusive Combine scan over the
//                segments (diagonal maps in (U, J)), giving the no-reset
//                state entering every segment; it overwrites the aggregates.
//   k_check      per (sample, segment, tile): re-walk from the carried state
//                with a no-crossing screen per inter-event interval
//                (screen_value).  Resets only lower V, so a sub-block of kSub
//                events whose no-reset trajectory passes every screen holds
//                no spike whatever happened before it; a flagged sub-block
//                reserves a pool entry and stores its entering state there.
//   k_resolve    per (sample, neuron) with flagged sub-blocks: walks only
//                those, in time order.  Staging waves walk each flagged
//                sub-block from its entering state (the no-reset state at
//                every interval start) and compute each interval's crossing
//                key, filling a ring of LDS windows ahead of the chain wave.
//                Spikes found so far lower V by a known decaying amount (the
//                reset deficit), which corrects the no-reset states exactly;
//                an interval crosses iff its key is at least the deficit's
//                current key (the interval rule of Sec. 3.2.2, one compare
//                per interval).  The spike time is solved by bracketed Newton
//                (Appendix D.1), V is hard-reset and the same interval is
//                tested again from the spike (Appendix E.2).
// The sequential baseline k_sequential (Appendix E.3) runs the same interval
// rule and root solve one event at a time per (sample, neuron).
#include "lif_common.hpp"
#include "lif_host.hpp"
#include "lif_walk.hpp"
#include "lif_reg.hpp"
#include <type_traits>

namespace lif {

// Pool of entering states: one entry (the no-reset (U, J) entering the
// sub-block) per flagged (sub-block, neuron), in per-sample slices.  The
// check pass reserves the entries (one atomic per wave) and writes them; the
// resolve pass rebuilds the sub-block's interval states from them.
constexpr uint32_t kNoSlot = 0xffffffffu;

// Mask word of a (sample, segment, neuron): the flagged sub-blocks in bits
// 0..3, the pool offset of the pair's first entry in bits 4..31.
constexpr int kMaskBits = 4;
static_assert(kSubPerSeg <= kMaskBits, "mask word layout");

// Search key of an interval whose crossing test is "reset deficit at its
// start <= crit" (crossing_data).  The deficit of the spikes so far is
// D(t) = dref e^{-(t - tref)/tm}, so at an interval that starts at t0 the
// test reads ln(crit) + t0/tm >= ln(dref) + tref/tm.  crit < 0 (never
// crosses) gives NaN, for which every comparison is false; crit = 0 gives
// -inf, which only the deficit of no spike at all (ln 0) reaches.
__device__ __forceinline__ double crossing_key(const Model& m, double crit, double t0)
{
    if (!(crit >= 0.0)) return __builtin_nan("");
    if (crit == 0.0) return -INFINITY;
    return log(crit) + t0 * m.inv_tm;
}

// A wait inside a workgroup that does not end within this many polls is an
// internal error (reported in the status words instead of waiting for ever).
constexpr int kSpinLimit = 1 << 22;

// Per-sample counters (pool use, work-list length) each take their
// own 128-byte line: many waves update them with atomics, and atomics on one
// line are serialised.
constexpr int kCtr = 32;

// ---------------------------------------------------------------------------
// k_prep
// ---------------------------------------------------------------------------
// Decay record of event k (gap to the previous event, or to t = 0).
__device__ __forceinline__ Decay make_decay(const Model& m, const float* __restrict__ t, int k)
{
    double dt = (double)t[k] - (k > 0 ? (double)t[k - 1] : 0.0);
    Decay d;
    d.A = exp(-dt * m.inv_tm);
    d.D = exp(-dt * m.inv_ts);
    d.C = unit_kernel(m, dt, d.A);
    d.lk = dt * m.inv_ktm;
    return d;
}

// Decays dec[B][E_pad] (identity maps past each sample's last event, so
// that the walks run whole sub-blocks), the composed maps (A, D) of every
// segment, and the reset of status words, counters and outputs (out_t is
// filled with +inf when given: the resolve pass writes only neurons that
// fire).
__global__ __launch_bounds__(256) void k_prep(const float* __restrict__ ev_t, const int32_t* __restrict__ ev_n,
                                              int B, int E_max, int E_pad, int S, Model m, Decay* __restrict__ dec,
                                              double2* __restrict__ segm, int32_t* __restrict__ status,
                                              uint32_t* __restrict__ counters, size_t n_counters,
                                              int32_t* __restrict__ out_n, uint32_t* __restrict__ listed, size_t nn,
                                              float* __restrict__ out_t, float* __restrict__ out_i,
                                              int32_t* __restrict__ out_k, size_t n_out)
{
    const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    if (tid < LIF_STATUS_WORDS) status[tid] = 0;
    for (size_t i = tid; i < n_counters; i += stride) counters[i] = 0u;
    for (size_t i = tid; i < nn; i += stride) {
        out_n[i] = 0;
        if (listed) listed[i] = 0u;
    }
    if (out_t) {
        for (size_t i = tid; i < n_out; i += stride) {
            out_t[i] = INFINITY;
            if (out_i) out_i[i] = 0.0f;
            if (out_k) out_k[i] = 0;
        }
    }
    const size_t nev = (size_t)B * (size_t)E_pad;
    for (size_t idx = tid; idx < nev; idx += stride) {
        const int b = (int)(idx / (size_t)E_pad), k = (int)(idx % (size_t)E_pad);
        Decay d{1.0, 1.0, 0.0, 0.0};
        if (k < clamp_count(ev_n[b], E_max)) d = make_decay(m, ev_t + (size_t)b * E_max, k);
        dec[idx] = d;
    }
    if (segm) {
        for (size_t idx = tid; idx < (size_t)B * S; idx += stride) {
            const int b = (int)(idx / (size_t)S), j = (int)(idx % (size_t)S);
            const int nb = clamp_count(ev_n[b], E_max), k0 = j * kSeg;
            double2 r = make_double2(1.0, 1.0);
            if (k0 < nb) {
                const float* tt = ev_t + (size_t)b * E_max;
                const double T = (double)tt[min(k0 + kSeg, nb) - 1] - (k0 > 0 ? (double)tt[k0 - 1] : 0.0);
                r = make_double2(exp(-T * m.inv_tm), exp(-T * m.inv_ts));
            }
            segm[idx] = r;
        }
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

// One event in eigen-coordinates: decay over the gap, then the jump.
template <int NPL>
__device__ __forceinline__ void step(double A, double D, const float (&w)[NPL], double (&U)[NPL], double (&J)[NPL])
{
#pragma unroll
    for (int i = 0; i < NPL; ++i) {
        const double x = (double)w[i];
        U[i] = fma(A, U[i], x);
        J[i] = fma(D, J[i], x);
    }
}

// One event in eigen-coordinates: decay over the gap, then the jump.
__device__ __forceinline__ void step1(double2 ad, float w, double& U, double& J)
{
    const double x = (double)w;
    U = fma(ad.x, U, x);
    J = fma(ad.y, J, x);
}

// Walk the n events of a group starting at e0 (n = kGrp on every group but
// a sample's last).
template <int NPL>
__device__ __forceinline__ void walk_grp(const double2* __restrict__ lad, int e0, int n, const float (&w)[kGrp][NPL],
                                         double (&U)[NPL], double (&J)[NPL])
{
    if (n >= kGrp) {
#pragma unroll
        for (int j = 0; j < kGrp; ++j) {
            const double2 ad = lad[e0 + j];
            step<NPL>(ad.x, ad.y, w[j], U, J);
        }
    } else {
#pragma unroll
        for (int j = 0; j < kGrp; ++j)
            if (j < n) {
                const double2 ad = lad[e0 + j];
                step<NPL>(ad.x, ad.y, w[j], U, J);
            }
    }
}

template <int NPL>
__global__ __launch_bounds__(kWave * kWalkWaves) void k_aggregate(
    const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src, const int32_t* __restrict__ ev_n, int E_max,
    int E_pad, const float* __restrict__ WT, int C_in, int N, int tiles, int S, int items, Model m,
    Decay* __restrict__ dec, double2* __restrict__ segm, double2* __restrict__ agg, int32_t* __restrict__ status,
    uint32_t* __restrict__ counters, size_t n_counters, uint32_t* __restrict__ listed, size_t nn,
    int32_t* __restrict__ out_n, float* __restrict__ out_t, float* __restrict__ out_i, int32_t* __restrict__ out_k,
    size_t n_out)
{
    {
        // resets for the later passes: status words, per-sample counters,
        // listed flags, and the outputs (the resolve pass writes only the
        // neurons that fire: counts 0, times +inf, currents and event
        // counts 0), grid-stride over every thread
        const size_t gt = (size_t)blockIdx.x * blockDim.x + threadIdx.x, gs = (size_t)gridDim.x * blockDim.x;
        if (gt < LIF_STATUS_WORDS) status[gt] = 0;
        for (size_t i = gt; i < n_counters; i += gs) counters[i] = 0u;
        for (size_t i = gt; i < nn; i += gs) {
            listed[i] = 0u;
            if (out_n) out_n[i] = 0;
        }
        if (out_t)
            for (size_t i = gt; i < n_out; i += gs) {
                out_t[i] = INFINITY;
                if (out_i) out_i[i] = 0.0f;
                if (out_k) out_k[i] = 0;
            }
    }
    __shared__ double2 s_ad[kWalkWaves][kSeg];
    WalkCoords c;
    if (!walk_coords<NPL>(items, tiles, S, ev_n, E_max, N, c)) return;
    double2* lad = s_ad[threadIdx.x / kWave];
    // the decays of the segment's events (identity past the sample's last
    // event); the first tile's wave stores them, and the segment's composed
    // map, for the later passes
    {
        const float* tt = ev_t + (size_t)c.b * E_max;
        Decay* dd = dec + (size_t)c.b * E_pad + c.k0;
#pragma unroll
        for (int h = 0; h < kSrcRegs; ++h) {
            const int e = h * kWave + c.lane;
            Decay dk{1.0, 1.0, 0.0, 0.0};
            if (c.k0 + e < c.nb) dk = make_decay(m, tt, c.k0 + e);
            lad[e] = make_double2(dk.A, dk.D);
            if (c.tile == 0) dd[e] = dk;
        }
        if (c.tile == 0 && c.lane == 0) {
            const double T = (double)tt[c.k0 + c.cnt - 1] - (c.k0 > 0 ? (double)tt[c.k0 - 1] : 0.0);
            segm[(size_t)c.b * S + c.seg] = make_double2(exp(-T * m.inv_tm), exp(-T * m.inv_ts));
        }
    }
    const Stage st = stage_segment(c, ev_src + (size_t)c.b * E_max + c.k0, nullptr, WT, C_in, N, lad, nullptr,
                                   nullptr);
    double U[NPL], J[NPL];
#pragma unroll
    for (int i = 0; i < NPL; ++i) U[i] = J[i] = 0.0;
    // Two weight buffers in alternation (no register copies): wa holds the
    // even and wb the odd groups.
    float wa[kGrp][NPL], wb[kGrp][NPL];
    load_grp<NPL>(st, 0, wa);
    for (int e0 = 0; e0 < c.cnt; e0 += 2 * kGrp) {
        load_grp<NPL>(st, e0 + kGrp, wb);
        walk_grp<NPL>(lad, e0, c.cnt - e0, wa, U, J);
        if (e0 + kGrp >= c.cnt) break;
        load_grp<NPL>(st, e0 + 2 * kGrp, wa);
        walk_grp<NPL>(lad, e0 + kGrp, c.cnt - e0 - kGrp, wb, U, J);
    }
    if (c.live) {
        const size_t row = ((size_t)c.b * S + c.seg) * N + c.n0;
#pragma unroll
        for (int i = 0; i < NPL; ++i) agg[row + i] = make_double2(U[i], J[i]);
    }
}

// Exclusive scan over segments of the Combine of Eq. affine in (U, J):
// s_in(j + 1) = M(T_j) s_in(j) + agg_j, s_in(0) = 0, where M(T_j) =
// diag(A_j, D_j) (segm).  A workgroup of kCarryWaves waves takes one
// (sample, 64-neuron tile); lanes are neurons and wave w the w-th contiguous
// range of at most kCarryBatch segments per round.  Each wave folds its range
// from the zero state (its aggregates loaded at once and kept), the range
// totals are combined across waves in LDS, and each wave walks its range
// again from its incoming state, writing the carries over the aggregates
// (each element is read before it is written, by the same wave).
constexpr int kCarryWaves = 8;
constexpr int kCarryBatch = 16;

__global__ __launch_bounds__(kWave * kCarryWaves) void k_carry(
    const int32_t* __restrict__ ev_n, int B, int E_max, int N, int tiles, int S, const double2* __restrict__ segm,
    const double2* agg, double2* carry)
{
    __shared__ double2 tot[kCarryWaves][kWave];      // range map b-part
    __shared__ double2 dec_tot[kCarryWaves];         // range map diagonal
    const int b = blockIdx.x / tiles, tile = blockIdx.x % tiles;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int n = tile * kWave + lane;
    const bool live = n < N;
    const int nc = live ? n : N - 1;
    const int nb = clamp_count(ev_n[b], E_max);
    const int Sb = (nb + kSeg - 1) / kSeg;
    double U = 0.0, J = 0.0;                         // state entering the current round
    for (int r0 = 0; r0 < Sb; r0 += kCarryWaves * kCarryBatch) {
        const int per = min(kCarryBatch, (Sb - r0 + kCarryWaves - 1) / kCarryWaves);
        const int j_lo = min(r0 + wave * per, Sb), j_hi = min(j_lo + per, Sb);
        double2 a[kCarryBatch], M[kCarryBatch];
#pragma unroll
        for (int j = 0; j < kCarryBatch; ++j) {
            const int jj = min(j_lo + j, Sb - 1);
            a[j] = agg[((size_t)b * S + jj) * N + nc];
            M[j] = segm[(size_t)b * S + jj];
        }
        // fold the range from zero
        double fU = 0.0, fJ = 0.0, pA = 1.0, pD = 1.0;
#pragma unroll
        for (int j = 0; j < kCarryBatch; ++j) {
            if (j_lo + j < j_hi) {
                fU = fma(M[j].x, fU, a[j].x);
                fJ = fma(M[j].y, fJ, a[j].y);
                pA *= M[j].x;
                pD *= M[j].y;
            }
        }
        tot[wave][lane] = make_double2(fU, fJ);
        if (lane == 0) dec_tot[wave] = make_double2(pA, pD);
        __syncthreads();
        // incoming state of this wave's range: the earlier ranges applied in order
        double iU = U, iJ = J;
        for (int w = 0; w < wave; ++w) {
            const double2 g = tot[w][lane], gd = dec_tot[w];
            iU = fma(gd.x, iU, g.x);
            iJ = fma(gd.y, iJ, g.y);
        }
        // state after the whole round (for the next round)
        for (int w = 0; w < kCarryWaves; ++w) {
            const double2 g = tot[w][lane], gd = dec_tot[w];
            U = fma(gd.x, U, g.x);
            J = fma(gd.y, J, g.y);
        }
        __syncthreads();
        // walk the range again, writing the carry entering each segment
#pragma unroll
        for (int j = 0; j < kCarryBatch; ++j) {
            if (j_lo + j < j_hi) {
                if (live) carry[((size_t)b * S + j_lo + j) * N + n] = make_double2(iU, iJ);
                iU = fma(M[j].x, iU, a[j].x);
                iJ = fma(M[j].y, iJ, a[j].y);
            }
        }
    }
}

// Screen of one group of intervals.  The coarse test bounds every interval
// of the group at once: with X = U - J at each interval start, the largest X
// and J over the group and the group's largest slope glk,
//   max_j [X_j + max(J_j - th, 0) lk_j] <= max X + max(max J - th, 0) glk,
// so a group that fails it holds no interval that passes screen_value.  The
// (rare) groups that pass are walked again from their entering state with
// the exact per-interval screen.  Returns the largest exact screen value
// (-inf when the coarse test rejects the group for every lane).
template <int NPL>
__device__ __forceinline__ void screen_grp(const Model& m, const double2* __restrict__ lad,
                                           const double* __restrict__ llk, double glk, int e0, int n,
                                           const float (&w)[kGrp][NPL], double (&U)[NPL], double (&J)[NPL],
                                           double (&z)[NPL])
{
    double Ug[NPL], Jg[NPL], xm[NPL], jm[NPL];
#pragma unroll
    for (int i = 0; i < NPL; ++i) {
        Ug[i] = U[i];
        Jg[i] = J[i];
        xm[i] = -INFINITY;
        jm[i] = -INFINITY;
    }
    auto track = [&](int j) {
        const double2 ad = lad[e0 + j];
#pragma unroll
        for (int i = 0; i < NPL; ++i) {
            xm[i] = fmax(xm[i], U[i] - J[i]);
            jm[i] = fmax(jm[i], J[i]);
        }
        step<NPL>(ad.x, ad.y, w[j], U, J);
    };
    if (n >= kGrp) {
#pragma unroll
        for (int j = 0; j < kGrp; ++j) track(j);
    } else {
#pragma unroll
        for (int j = 0; j < kGrp; ++j)
            if (j < n) track(j);
    }
    bool pass = false;
#pragma unroll
    for (int i = 0; i < NPL; ++i) pass |= fma(fmax(jm[i] - m.th, 0.0), glk, xm[i]) >= m.thk_lo;
    if (__ballot(pass) == 0ull) return;
#pragma unroll
    for (int j = 0; j < kGrp; ++j) {
        if (j < n) {
            const double lk = llk[e0 + j];
            const double2 ad = lad[e0 + j];
#pragma unroll
            for (int i = 0; i < NPL; ++i) z[i] = fmax(z[i], screen_value(m, Ug[i], Jg[i], lk));
            step<NPL>(ad.x, ad.y, w[j], Ug, Jg);
        }
    }
}

// Re-walk from the carried no-reset state with the no-crossing screen on
// every interval: the interval before each event of the sub-block and, in
// the sub-block holding the sample's last event, the open interval after it
// (up to t_end).  A flagged (sub-block, neuron) sets a bit in the neuron's
// sub-block mask of the segment; the entering state (U, J) of every
// sub-block is kept in LDS until the pool entries are reserved.  At the end
// of the item the wave reserves entries for all its flagged sub-blocks with
// one atomic on the sample's pool counter, in lane order, so that the
// entries of one (segment, neuron) are consecutive: the mask word of the pair
// holds the sub-block bits and the pool offset of its first entry, and the
// entry of a flagged sub-block is that offset plus the number of flagged
// sub-blocks before it (none past the pool capacity: the resolve pass then
// rebuilds that sub-block's entering state from the segment's carried
// state).  The wave writes the entering states; the first segment to flag a
// neuron appends it to the sample's work list.
__global__ __launch_bounds__(kWave * kWalkWaves) void k_check(
    const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src, const int32_t* __restrict__ ev_n, int E_max,
    int E_pad, const float* __restrict__ WT, int C_in, int N, int tiles, int S, int items, Model m,
    const Decay* __restrict__ dec, const double2* __restrict__ carry, uint32_t* __restrict__ mask,
    double2* __restrict__ pool,
    uint32_t* __restrict__ pool_count, uint32_t pool_cap, uint32_t* __restrict__ listed,
    uint32_t* __restrict__ work, uint32_t* __restrict__ nwork)
// work: per-sample lists of the neurons with flagged sub-blocks (capacity N
// each); nwork: per-sample list lengths.
{
    constexpr int NPL = 1;                  // one neuron per lane (occupancy)
    __shared__ double2 s_ad[kWalkWaves][kSeg];
    __shared__ double s_lk[kWalkWaves][kSeg];
    __shared__ double s_gk[kWalkWaves][kGrpPerSeg];
    __shared__ double2 s_ent[kWalkWaves][kSubPerSeg][kWave];   // entering state of each sub-block
    WalkCoords c;
    if (!walk_coords<NPL>(items, tiles, S, ev_n, E_max, N, c)) return;
    const int lane = c.lane;
    const int wv = threadIdx.x / kWave;
    double2* lad = s_ad[wv];
    double* llk = s_lk[wv];
    double* lgk = s_gk[wv];
    const Stage st = stage_segment(c, ev_src + (size_t)c.b * E_max + c.k0, dec + (size_t)c.b * E_pad + c.k0, WT,
                                   C_in, N, lad, llk, lgk);
    const size_t row = ((size_t)c.b * S + c.seg) * N + c.n0;
    const unsigned long long below = (1ull << lane) - 1ull;
    double U[NPL], J[NPL];
#pragma unroll
    for (int i = 0; i < NPL; ++i) {
        const double2 s0 = carry[row + i];
        U[i] = s0.x;
        J[i] = s0.y;
    }
    uint32_t msk[NPL];
#pragma unroll
    for (int i = 0; i < NPL; ++i) msk[i] = 0u;
    // The open interval after the sample's last event, up to t_end.
    const bool last_seg = c.k0 + c.cnt == c.nb;
    const double open_lk = last_seg ? (m.t_end - (double)ev_t[(size_t)c.b * E_max + c.nb - 1]) * m.inv_ktm : 0.0;
    // Two weight buffers in alternation: wa holds the first and wb the second
    // group of each sub-block.
    float wa[kGrp][NPL], wb[kGrp][NPL];
    load_grp<NPL>(st, 0, wa);
    for (int q = 0; q < kSubPerSeg; ++q) {
        const int q0 = q * kSub;
        if (q0 >= c.cnt) break;
        double U0[NPL], J0[NPL], z[NPL];
#pragma unroll
        for (int i = 0; i < NPL; ++i) {
            U0[i] = U[i];
            J0[i] = J[i];
            z[i] = -INFINITY;
        }
        load_grp<NPL>(st, q0 + kGrp, wb);
        screen_grp<NPL>(m, lad, llk, lgk[2 * q], q0, c.cnt - q0, wa, U, J, z);
        if (q0 + kGrp < c.cnt) {
            load_grp<NPL>(st, q0 + kSub, wa);
            screen_grp<NPL>(m, lad, llk, lgk[2 * q + 1], q0 + kGrp, c.cnt - q0 - kGrp, wb, U, J, z);
        }
        if (last_seg && q0 + kSub >= c.cnt && open_lk > 0.0) {
#pragma unroll
            for (int i = 0; i < NPL; ++i)
                z[i] = fmax(z[i], J[i] > m.th ? fma(J[i] - m.th, open_lk, U[i] - J[i]) : U[i] - J[i]);
        }
        s_ent[wv][q][lane] = make_double2(U0[0], J0[0]);
#pragma unroll
        for (int i = 0; i < NPL; ++i)
            if (c.live && z[i] >= m.thk_lo) msk[i] |= 1u << q;
    }
    // Pool entries of the wave's flagged sub-blocks: one reservation, slots
    // in lane order (exclusive prefix sum of the per-lane counts).
    {
        uint32_t mine = 0;
#pragma unroll
        for (int i = 0; i < NPL; ++i) mine += (uint32_t)__popc(msk[i]);
        uint32_t ex = mine;
#pragma unroll
        for (int off = 1; off < kWave; off <<= 1) {
            const uint32_t v = (uint32_t)__shfl_up((int)ex, off, kWave);
            if (lane >= off) ex += v;
        }
        const uint32_t total = (uint32_t)__shfl((int)ex, kWave - 1, kWave);
        ex -= mine;
        uint32_t base = 0;
        if (total) {
            if (lane == 0) base = atomicAdd(&pool_count[(size_t)c.b * kCtr], total);
            base = (uint32_t)__shfl((int)base, 0, kWave) + ex;
        }
#pragma unroll
        for (int i = 0; i < NPL; ++i) {
            if (c.live) mask[row + i] = msk[i] | (base << kMaskBits);
            for (uint32_t mm = msk[i]; mm; mm &= mm - 1u) {
                if (base < pool_cap) pool[(size_t)c.b * pool_cap + base] = s_ent[wv][__builtin_ctz(mm)][lane];
                ++base;
            }
        }
    }
    // Work list of the sample: the first segment to flag a neuron appends it
    // (one OR per flagged neuron, one counter update per wave).
    bool want[NPL], first[NPL];
    unsigned long long wm = 0ull;
#pragma unroll
    for (int i = 0; i < NPL; ++i) {
        want[i] = c.live && msk[i] != 0u;
        wm |= __ballot(want[i]);
    }
    if (wm) {
        unsigned long long fmk[NPL];
        uint32_t tot = 0;
#pragma unroll
        for (int i = 0; i < NPL; ++i) {
            first[i] = false;
            if (want[i]) first[i] = atomicOr(&listed[(size_t)c.b * N + c.n0 + i], 1u) == 0u;
            fmk[i] = __ballot(first[i]);
            tot += (uint32_t)__popcll(fmk[i]);
        }
        if (tot) {
            uint32_t wbase = 0;
            if (lane == 0) wbase = atomicAdd(&nwork[(size_t)c.b * kCtr], tot);
            wbase = (uint32_t)__shfl((int)wbase, 0, kWave);
            uint32_t before = 0;
#pragma unroll
            for (int i = 0; i < NPL; ++i) {
                if (first[i])
                    work[(size_t)c.b * N + wbase + before + (uint32_t)__popcll(fmk[i] & below)] =
                        (uint32_t)((size_t)c.b * N + c.n0 + i);
                before += (uint32_t)__popcll(fmk[i]);
            }
        }
    }
}
// Crossing data of one interval of length L that starts in the no-reset
// state (V0, I0) and ends with V1 (A, D: its decays): the interval reaches
// the threshold iff the reset deficit at its start is <= crit (crit < 0:
// never), by interval_max's test D a <= g; the spike then lies in
// (lo, hi] with F(hi) = fhi - deficit.  Zero-length intervals never cross.
// Floating-point contraction is off here and in interval_max, so every
// inlined copy performs the same IEEE operations.
__device__ __forceinline__ void crossing_data(const Model& m, double V0, double I0, double V1, double L, double A,
                                              double D, double& crit, double& hi, double& fhi)
{
#pragma clang fp contract(off)
    crit = -1.0;
    hi = 0.0;
    fhi = -INFINITY;
    if (!(L > 0.0)) return;
    const IntervalMax im = interval_max(m, V0, I0, V1, L, A, D);
    if (im.g >= 0.0) crit = im.a > 0.0 ? im.g / im.a : INFINITY;
    hi = im.hi;
    fhi = im.Fhi;
}

// Crossing data of the open interval (t_last, t_end] after a sample's last
// event, from the state (V, I) right after it.
__device__ __forceinline__ void open_interval_data(const Model& m, double V, double I, double L, double& crit,
                                                   double& hi, double& fhi)
{
    double A = 0.0, D = 0.0, V1 = 0.0;
    if (!isinf(L)) {
        A = exp(-L * m.inv_tm);
        D = exp(-L * m.inv_ts);
        V1 = V * A + unit_kernel(m, L, A) * I;
    }
    crossing_data(m, V, I, V1, L, A, D, crit, hi, fhi);
}

__device__ __forceinline__ int rl_int(int v, int l) { return __builtin_amdgcn_readlane(v, l); }

__device__ __forceinline__ double rl_double(double v, int l)
{
    unsigned long long u = (unsigned long long)__double_as_longlong(v);
    unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)u, l);
    unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(u >> 32), l);
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// ---------------------------------------------------------------------------
// Resolve pass: one workgroup of four waves per neuron that has flagged
// sub-blocks (the work lists of the check pass).  Intervals outside flagged
// sub-blocks provably hold no spike.  The flagged sub-blocks are taken in
// time order:
//   * Candidate list: per chunk of kChunkEv events, the sub-block masks (two
//     segments per lane) are compacted into a time-ordered list in LDS with
//     one wave prefix sum, with the pool slot of every candidate.
//   * Windows of kWinCand candidates (kWinIv intervals) in a ring of kRing
//     LDS buffers: the staging waves (waves 1..3, windows in turn) walk the
//     window's sub-blocks and fill its buffer while the chain wave (wave 0)
//     works on an earlier one; a ready word per buffer and a consumed count
//     hand the buffers over (no barrier per window).
//   * The chain searches a window 64 intervals at a time: interval i crosses
//     iff key_i >= K, the key of the current reset deficit (crossing_key), so
//     one ballot finds the earliest crossing.  Its spike time is solved
//     wave-uniform, the deficit and K are raised, and the search resumes at
//     the same interval (a second spike in it, App. E.2 restart).
//   * The open interval after the sample's last event is one more slot of
//     the window holding the sample's last sub-block.
//   * Spikes are buffered in LDS and written out kWave at a time.
// ---------------------------------------------------------------------------
constexpr int kChunkEv = 8192;                   // events per chunk of the candidate list
constexpr int kChunkSeg = kChunkEv / kSeg;       // segments per chunk
constexpr int kSegPerLane = kChunkSeg / kWave;   // mask words per lane
static_assert(kChunkSeg % kWave == 0 && kSubPerSeg <= 8, "chunk layout; 3-bit sub-block field of a candidate");
constexpr int kCandCap = kChunkSeg * kSubPerSeg; // candidates of one chunk
constexpr int kCandPerStep = kWave / kSub;       // candidates per 64 intervals
constexpr int kWinCand = kCandPerStep;           // candidates per window (one interval per lane)
constexpr int kWinIv = kWinCand * kSub;          // intervals per window
static_assert(kWinIv == kWave, "one window interval per lane");
constexpr int kOpenIv = kWinIv;                  // window slot of the open interval
constexpr int kRing = 8;                         // window buffers
constexpr int kResolveWaves = 4;                 // the chain wave and three staging waves

struct WinBuf {
    double key[kWinIv + 1];                      // crossing key (NaN: no interval)
    double v0[kWinIv + 1], i0[kWinIv + 1];       // no-reset (V, I) at the interval start
    float t0[kWinIv + 1];                        // interval start (time of the event before it; 0 for the first)
    float t1[kWinIv + 1];                        // interval end (its closing event's time)
};

struct ResolveLds {
    uint32_t cand[kCandCap];                     // (segment in chunk << 3) | sub-block
    uint32_t slot[kCandCap];                     // pool slot of each candidate (kNoSlot: none)
    WinBuf win[kRing];
    double sp_t0[kWave], sp_y[kWave];            // spike buffer: interval start, e^{-u/tm},
    float si[kWave];                             // I at the spike,
    int32_t sk[kWave];                           // events consumed before the spike
    double open_len;                             // length of the open interval (t_end - last event)
    int ntot;                                    // candidates of the chunk (chain wave -> both)
    int ready[kRing];                            // 1 + window index staged in each buffer
    double kmax[kRing];                          // largest key of each buffer's window (NaN keys left out)
    int consumed;                                // windows the chain has finished
    int stop;                                    // the chain reached s_max
    unsigned long long kpub;                     // bits of the chain's current deficit key K
};

__device__ __forceinline__ int lds_load(const int* p)
{
    return __hip_atomic_load(const_cast<int*>(p), __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ void lds_store(int* p, int v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Entering no-reset state of sub-block kq0 (of the segment whose first
// event is k0) from the segment's carried state (U, J), for a sub-block past
// the pool's capacity, by the whole wave: lane e loads event k0 + e's weight
// and decays, and every lane follows the same serial walk over events k0 ..
// kq0 - 1 with those values broadcast (the check pass's operations, so the
// state has the bits a pool entry would hold).  Wave-uniform result.
__device__ double2 rebuild_entry(double U, double J, int k0, int kq0, int n, int N, int C_in,
                                 const int32_t* __restrict__ src, const Decay* __restrict__ d,
                                 const float* __restrict__ WT)
{
    const int lane = (int)threadIdx.x % kWave;
    const int ne = kq0 - k0;
    float we = 0.0f;
    double A = 1.0, D = 1.0;
    if (lane < ne) {
        we = WT[(size_t)clamp_src(src[k0 + lane], C_in) * (size_t)N + n];
        const Decay dk = d[k0 + lane];
        A = dk.A;
        D = dk.D;
    }
    for (int e = 0; e < ne; ++e) {
        const float w = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, we), e));
        step1(make_double2(rl_double(A, e), rl_double(D, e)), w, U, J);
    }
    return make_double2(U, J);
}

// Lane E's value of the calling lane's row of 16 lanes (DPP row broadcast).
template <int E>
__device__ __forceinline__ int row_bcast(int v)
{
    return __builtin_amdgcn_update_dpp(0, v, 0x150 + E, 0xf, 0xf, false);
}

template <int E>
__device__ __forceinline__ double row_bcast(double v)
{
    const unsigned long long u = (unsigned long long)__double_as_longlong(v);
    const unsigned lo = (unsigned)row_bcast<E>((int)(unsigned)u), hi = (unsigned)row_bcast<E>((int)(unsigned)(u >> 32));
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// The value of lane j - Dist of the calling lane's row of 16 lanes (DPP
// row shift); lanes j < Dist get fill.
template <int Dist>
__device__ __forceinline__ double row_shr(double v, double fill)
{
    const unsigned long long u = (unsigned long long)__double_as_longlong(v);
    const unsigned long long f = (unsigned long long)__double_as_longlong(fill);
    const unsigned lo = (unsigned)__builtin_amdgcn_update_dpp((int)(unsigned)f, (int)(unsigned)u, 0x110 + Dist, 0xf,
                                                              0xf, false);
    const unsigned hi = (unsigned)__builtin_amdgcn_update_dpp((int)(unsigned)(f >> 32), (int)(unsigned)(u >> 32),
                                                              0x110 + Dist, 0xf, 0xf, false);
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// One step of the row's inclusive scan of event maps in (U, J): lane j's map
// (a, b) (x -> a x + b) composed after the map of lane j - Dist.
template <int Dist>
__device__ __forceinline__ void scan_step(double& aU, double& bU, double& aJ, double& bJ)
{
    const double paU = row_shr<Dist>(aU, 1.0), pbU = row_shr<Dist>(bU, 0.0);
    const double paJ = row_shr<Dist>(aJ, 1.0), pbJ = row_shr<Dist>(bJ, 0.0);
    bU = fma(aU, pbU, bU);
    aU *= paU;
    bJ = fma(aJ, pbJ, bJ);
    aJ *= paJ;
}

// The no-reset states of a sub-block's intervals from its entering state u0
// (one row of 16 lanes, lane j holding event j of the sub-block with decays
// (A, D) and weight w): the maps of events 0 .. j composed by a log-depth
// scan within the row (App. B: the maps form a semigroup), so lane j gets
// the state at the start of its interval (after event j - 1) and after its
// event.
__device__ __forceinline__ void row_states(double2 u0, double A, double D, float w, double& U0, double& J0,
                                           double& U1, double& J1)
{
    double aU = A, bU = (double)w, aJ = D, bJ = (double)w;
    scan_step<1>(aU, bU, aJ, bJ);
    scan_step<2>(aU, bU, aJ, bJ);
    scan_step<4>(aU, bU, aJ, bJ);
    scan_step<8>(aU, bU, aJ, bJ);
    U1 = fma(aU, u0.x, bU);
    J1 = fma(aJ, u0.y, bJ);
    U0 = fma(row_shr<1>(aU, 1.0), u0.x, row_shr<1>(bU, 0.0));
    J0 = fma(row_shr<1>(aJ, 1.0), u0.y, row_shr<1>(bJ, 0.0));
}

// A value <= e^x for the staging screen: the float exponential (relative
// error below 2^-16 for |x| <= 88, argument rounding included) scaled by
// 1 - 2^-10; 0 below the float range and at most FLT_MAX above it (beyond
// it the deficit exceeds any state the screen could pass).
__device__ __forceinline__ double exp_lower(double x)
{
    return (1.0 - 0x1p-10) * (double)fminf(__expf((float)x), 3.0e38f);
}

// A staging wave's window: candidates c0 .. c0 + kWinCand - 1 of the chunk,
// lane l taking interval j = l % kSub of candidate c0 + l / kSub.  Every lane
// loads its own interval's closing event (source, decays, times) and its
// candidate's entering state (stage_load, issued before the wait for the
// window's buffer), then its weight; the 16
// lanes of a candidate (one row) take the no-reset states of the sub-block by
// a scan of its event maps (row_states), lane j the state at its interval's
// start (after event j - 1) and end, and the interval's crossing key.  Candidates past the pool's capacity take
// their entering state from rebuild_entry.  open_last: the window holds the
// sample's last sub-block, and the open interval after its last event is
// staged too.
struct StageIn {
    int k, sc;
    bool ok;
    uint32_t slot;
    double A, D;
    float ta, tb;
    double2 u0;
};

__device__ __forceinline__ StageIn stage_load(const ResolveLds& sh, int c0, int tot, int seg0, int nb,
                                              const float* __restrict__ tt, const int32_t* __restrict__ src,
                                              const Decay* __restrict__ d, const double2* __restrict__ pool)
{
    const int lane = (int)threadIdx.x % kWave;
    const int j = lane % kSub, r = lane / kSub;
    const int c = c0 + r;
    const int cc = min(c, tot - 1);
    const uint32_t cw = sh.cand[cc];
    StageIn in;
    in.slot = sh.slot[cc];
    const int kq = (seg0 + (int)(cw >> 3)) * kSeg + (int)(cw & 7u) * kSub;
    in.ok = c < tot && kq + j < nb;
    in.k = min(kq + j, nb - 1);
    in.sc = src[in.k];
    const Decay dk = d[in.k];
    in.A = dk.A;
    in.D = dk.D;
    in.ta = tt[max(in.k - 1, 0)];
    in.tb = tt[in.k];
    in.u0 = pool[in.slot != kNoSlot ? in.slot : 0u];    // the pool holds at least one entry
    return in;
}

__device__ __forceinline__ void stage_window(ResolveLds& sh, WinBuf& w, const Model& m, const StageIn& in, int c0,
                                             int tot, int seg0, int b, int n, int nb, int S, int N, int C_in,
                                             const int32_t* __restrict__ src, const Decay* __restrict__ d,
                                             const float* __restrict__ WT, const double2* __restrict__ carry,
                                             bool open_last, double& kmax)
{
    const int lane = (int)threadIdx.x % kWave;
    const int r = lane / kSub;
    const int c = c0 + r;
    const int k = in.k, sc = in.sc;
    const bool ok = in.ok;
    const double2 ad = make_double2(in.A, in.D);
    const float ta = in.ta, tb = in.tb;
    double2 u0 = in.u0;
    const float wv = WT[(size_t)clamp_src(sc, C_in) * (size_t)N + n];
    if (__ballot(c < tot && in.slot == kNoSlot)) {
        const int nc = min(kWinCand, tot - c0);
        for (int x = 0; x < nc; ++x) {
            if (sh.slot[c0 + x] != kNoSlot) continue;
            const uint32_t cx = sh.cand[c0 + x];
            const int seg = seg0 + (int)(cx >> 3);
            const double2 cs = carry[((size_t)b * S + seg) * N + n];
            const double2 e = rebuild_entry(cs.x, cs.y, seg * kSeg, seg * kSeg + (int)(cx & 7u) * kSub, n, N, C_in,
                                            src, d, WT);
            if (x == r) u0 = e;
        }
    }
    double U0, J0, U, J;
    row_states(u0, ad.x, ad.y, wv, U0, J0, U, J);
    const double V0 = v_of(m, U0, J0), I0 = J0;
    const double V1 = v_of(m, U, J);
    const double t0 = k > 0 ? (double)ta : 0.0, t1 = (double)tb;
    // The deficit of the spikes the chain has found so far, decayed to the
    // interval's start, bounds the true deficit there from below (the chain
    // works on earlier windows, and later spikes only add to it), so the
    // no-crossing screen of the true state is safe with it (with a lower
    // bound of that deficit, exp_lower).  Most intervals of a neuron that has
    // fired fail it; the crossing key is computed only when some lane passes.
    const double Kp = __longlong_as_double((long long)__hip_atomic_load(&sh.kpub, __ATOMIC_RELAXED,
                                                                        __HIP_MEMORY_SCOPE_WORKGROUP));
    const double L = t1 - t0;
    const bool maybe = ok && L > 0.0 &&
                       (V0 - exp_lower(Kp - t0 * m.inv_tm)) + (I0 > m.th ? (I0 - m.th) * (L * m.inv_tm) : 0.0) >=
                           m.th_lo;
    double key = __builtin_nan("");
    double crit, hi, fhi;
    if (__ballot(maybe)) {
        crossing_data(m, V0, I0, V1, L, ad.x, ad.y, crit, hi, fhi);
        if (maybe) key = crossing_key(m, crit, t0);
    }
    w.key[lane] = key;
    double km = key;
    w.v0[lane] = V0;
    w.i0[lane] = I0;
    w.t0[lane] = k > 0 ? ta : 0.0f;
    w.t1[lane] = tb;
    if (open_last && ok && k == nb - 1) {
        // the open interval after the sample's last event (the same screen)
        const double Lo = m.t_end - t1;
        const bool mo = Lo > 0.0 &&
                        (V1 - exp_lower(Kp - t1 * m.inv_tm)) + (J > m.th ? (J - m.th) * (Lo * m.inv_tm) : 0.0) >=
                            m.th_lo;
        double ko = __builtin_nan("");
        if (mo) {
            open_interval_data(m, V1, J, Lo, crit, hi, fhi);
            ko = crossing_key(m, crit, t1);
        }
        w.key[kOpenIv] = ko;
        w.v0[kOpenIv] = V1;
        w.i0[kOpenIv] = J;
        w.t0[kOpenIv] = tb;
        sh.open_len = m.t_end - t1;
        km = fmax(km, w.key[kOpenIv]);
    }
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) km = fmax(km, __shfl_xor(km, off, kWave));
    if (lane == 0) kmax = km;
}

// Wave-uniform resolve state of one neuron: the reset deficit of the spikes
// so far is D(t) = dref e^{-(t - tref)/tm} for t after the latest spike,
// with tref the start of the interval that spike lies in (the deficit is
// carried in that interval's frame), and K = ln(dref) + tref/tm its key.
struct Chain {
    int ns;              // spikes so far
    double dref, tref, K;
    double ylast;        // e^{-u/tm} of the latest spike (its offset u in its interval)
    int lastw, lasti;    // window and interval of the latest spike
    bool capped;
};

// Spikes [from, to) from the LDS buffer to the outputs (coalesced); the
// spike times t0 - tm ln y are taken here, 64 at a time, off the chain.
__device__ __forceinline__ void flush_spikes(ResolveLds& sh, const Model& m, int from, int to, float* __restrict__ st,
                                             float* __restrict__ si, int32_t* __restrict__ sk)
{
    const int lane = (int)threadIdx.x % kWave;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (from + lane < to) {
        const int q = (from + lane) % kWave;
        st[from + lane] = (float)(sh.sp_t0[q] - m.tm * log(sh.sp_y[q]));
        if (si) si[from + lane] = sh.si[q];
        if (sk) sk[from + lane] = sh.sk[q];
    }
    __builtin_amdgcn_wave_barrier();
}

// The spike in window interval i (the earliest crossing the search found):
// the deficit at the interval start, the spike time (polynomial solve when
// tau_m / tau_s is an integer plus one, else bracketed Newton on the
// interval's closed-form maximum), the spike into the LDS buffer, and the
// raised deficit in the interval's frame.  Returns false at s_max.
template <int PI>
__device__ bool spike_at(ResolveLds& sh, const WinBuf& w, const Model& m, int i, int wg, int c0, int seg0, int nb,
                         Chain& ch, float* __restrict__ st, float* __restrict__ si, int32_t* __restrict__ sk)
{
    const int lane = (int)threadIdx.x % kWave;
    const double V0 = rl_double(w.v0[i], 0), I0 = rl_double(w.i0[i], 0);
    const double t0 = (double)__builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, w.t0[i])));
    const double Dk = ch.ns > 0 ? ch.dref * exp(-(t0 - ch.tref) * m.inv_tm) : 0.0;
    const double ylo = (ch.ns > 0 && ch.lastw == wg && ch.lasti == i) ? ch.ylast : 1.0;
    const double kI = m.kappa * I0, c0v = V0 - Dk + kI;
    double y = 0.0, E1 = 0.0, E2 = 0.0;
    bool ok = false;
    if constexpr (PI > 0) {
        ok = root_poly<PI>(m, c0v, kI, ylo, y);
        if (ok) E2 = ipow<PI>(y);
    }
    if (ok) {
        E1 = rcp_refined(y);
    } else {
        // the exponential solve brackets the root in [0, hi] with the
        // interval's closed-form maximum (interval_max)
        const double L = i == kOpenIv ? sh.open_len : (double)w.t1[i] - t0;
        double A = 0.0, D = 0.0, V1 = 0.0;
        if (!isinf(L)) {
            A = exp(-L * m.inv_tm);
            D = exp(-L * m.inv_ts);
            V1 = V0 * A + unit_kernel(m, L, A) * I0;
        }
        const IntervalMax im = interval_max(m, V0, I0, V1, L, A, D);
        root_h(m, c0v, kI, 0.0, V0 - m.th - Dk, im.hi, im.Fhi - Dk, &E1, &E2, nullptr);
        y = rcp_refined(E1);
    }
    int kev = nb;
    if (i != kOpenIv) {
        const uint32_t cw = sh.cand[c0 + i / kSub];
        kev = (seg0 + (int)(cw >> 3)) * kSeg + (int)(cw & 7u) * kSub + i % kSub;
    }
    if (lane == 0) {
        const int q = ch.ns % kWave;
        sh.sp_t0[q] = t0;
        sh.sp_y[q] = y;
        sh.si[q] = (float)(I0 * (E2 * y));
        sh.sk[q] = kev;
    }
    const double Dnew = Dk + m.dth * E1;
    ch.dref = Dnew;
    ch.tref = t0;
    ch.K = log(Dnew) + t0 * m.inv_tm;
    if (lane == 0)
        __hip_atomic_store(&sh.kpub, (unsigned long long)__double_as_longlong(ch.K), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_WORKGROUP);
    ch.ylast = y;
    ch.lastw = wg;
    ch.lasti = i;
    ++ch.ns;
    if (ch.ns % kWave == 0) flush_spikes(sh, m, ch.ns - kWave, ch.ns, st, si, sk);
    if (ch.ns >= m.s_max) {
        ch.capped = true;
        return false;
    }
    return true;
}

// The chain wave's work on one window: its n_iv intervals (one per lane),
// then (open_last) the open interval; one call site of the spike solve keeps
// the kernel's code small.
template <int PI>
__device__ __forceinline__ void chain_window(ResolveLds& sh, const WinBuf& w, const Model& m, int wg, int c0, int n_iv,
                                             bool open_last, int seg0, int nb, Chain& ch, float* __restrict__ st,
                                             float* __restrict__ si, int32_t* __restrict__ sk)
{
    const int lane = (int)threadIdx.x % kWave;
    const int nh = n_iv > 0 ? 1 : 0;
    const int hend = open_last ? nh + 1 : nh;
    const double kb = w.key[lane], ko = w.key[kOpenIv];
    for (int h = 0; h < hend; ++h) {
        const bool open = h == nh;
        const double key = open ? ko : kb;
        int from = 0;
        for (;;) {
            const unsigned long long cm = __ballot((open ? lane == 0 : lane >= from) && key >= ch.K);
            if (cm == 0ull) break;
            const int kl = __ffsll((long long)cm) - 1;
            if (!spike_at<PI>(sh, w, m, open ? kOpenIv : h * kWave + kl, wg, c0, seg0, nb, ch, st, si, sk)) return;
            from = kl;
        }
    }
}

// Both waves of the workgroup call this for the same neuron and pass the
// same barriers (one per chunk; candidate counts and the stop flag pass
// through LDS).  Returns the spike count on the chain wave, 0 on the
// staging wave.
template <int PI>
__device__ int resolve_neuron(ResolveLds& sh, int b, int n, const float* __restrict__ ev_t,
                              const int32_t* __restrict__ ev_src, const int32_t* __restrict__ ev_n, int E_max,
                              const float* __restrict__ WT, int C_in, int N, int E_pad, int S, const Model& m,
                              const Decay* __restrict__ dec, const double2* __restrict__ carry,
                              const uint32_t* __restrict__ mask, uint32_t pool_cap, const double2* __restrict__ pool,
                              float* __restrict__ out_t, int32_t* __restrict__ out_n, float* __restrict__ out_i,
                              int32_t* __restrict__ out_k, int32_t* __restrict__ status)
{
    const int lane = (int)threadIdx.x % kWave;
    const int wv = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
    const bool chain = wv == 0;               // wave 0 resolves, waves 1.. stage (wave-uniform)
    // the chain is the critical path: its instructions go first on its SIMD
    if (chain) __builtin_amdgcn_s_setprio(3);
    // a wait that does not end within kSpinLimit polls is an internal error:
    // it is reported and the neuron is stopped instead of waiting for ever
    auto give_up = [&]() {
        if (lane == 0) atomicOr(&status[LIF_ST_FLAGS], LIF_WARN_INTERNAL);
        lds_store(&sh.stop, 1);
    };
    if (threadIdx.x == 0) {
        sh.consumed = 0;
        sh.stop = 0;
        sh.kpub = (unsigned long long)__double_as_longlong(-INFINITY);
        for (int r = 0; r < kRing; ++r) sh.ready[r] = 0;
    }
    // the first chunk's mask words are loaded together with the event count
    // (words past the sample's segments are dropped below)
    uint32_t mw[kSegPerLane];
#pragma unroll
    for (int h = 0; h < kSegPerLane; ++h) {
        const int sj = lane * kSegPerLane + h;
        mw[h] = chain && sj < S ? mask[((size_t)b * S + sj) * N + n] : 0u;
    }
    const int nb = __builtin_amdgcn_readfirstlane(clamp_count(ev_n[b], E_max));
    const float* tt = ev_t + (size_t)b * E_max;
    const int32_t* src = ev_src + (size_t)b * E_max;
    const Decay* d = dec + (size_t)b * E_pad;
    const size_t idx = (size_t)b * N + n;
    float* st = out_t + idx * (size_t)m.s_max;
    float* si = out_i ? out_i + idx * (size_t)m.s_max : nullptr;
    int32_t* sk = out_k ? out_k + idx * (size_t)m.s_max : nullptr;
    const int Sb = (nb + kSeg - 1) / kSeg;
    const bool has_open = __builtin_amdgcn_readfirstlane(nb > 0 && m.t_end > (double)tt[max(nb - 1, 0)] ? 1 : 0) != 0;
    __syncthreads();                          // the ring is reset

    Chain ch{0, 0.0, 0.0, -INFINITY, 1.0, -1, -1, false};
    int wbase = 0;                            // windows of earlier chunks
    bool stop = false;
    for (int seg0 = 0; seg0 < Sb && !stop; seg0 += kChunkSeg) {
        // ---- this chunk's flagged sub-blocks as a time-ordered list, with
        // slots; lane l takes segments seg0 + kSegPerLane l + h
        if (chain) {
            uint32_t mv[kSegPerLane];
            int pc = 0;
#pragma unroll
            for (int h = 0; h < kSegPerLane; ++h) {
                const int sj = seg0 + lane * kSegPerLane + h;
                if (seg0 > 0) mw[h] = sj < Sb ? mask[((size_t)b * S + sj) * N + n] : 0u;
                mv[h] = sj < Sb ? (mw[h] & ((1u << kSubPerSeg) - 1u)) : 0u;
                pc += __popc(mv[h]);
            }
            int ex = pc;
#pragma unroll
            for (int off = 1; off < kWave; off <<= 1) {
                const int v = __shfl_up(ex, off, kWave);
                if (lane >= off) ex += v;
            }
            const int ctot = rl_int(ex, kWave - 1);
            ex -= pc;
            // candidates and their pool slots (consecutive per segment)
            int o = ex;
#pragma unroll
            for (int h = 0; h < kSegPerLane; ++h) {
                uint32_t mm = mv[h], rel = mw[h] >> kMaskBits;
                while (mm) {
                    sh.cand[o] = ((uint32_t)(lane * kSegPerLane + h) << 3) | (uint32_t)__builtin_ctz(mm);
                    sh.slot[o] = rel < pool_cap ? (uint32_t)b * pool_cap + rel : kNoSlot;
                    ++o;
                    ++rel;
                    mm &= mm - 1u;
                }
            }
            if (lane == 0) sh.ntot = ctot;
        }
        __syncthreads();
        const int tot = __builtin_amdgcn_readfirstlane(sh.ntot);
        const int nwin = (tot + kWinCand - 1) / kWinCand;
        if (tot > 0) {
            // the open interval is taken after the window holding the sample's
            // last sub-block, when that sub-block is flagged (it is the last
            // candidate of the last chunk)
            const uint32_t cwl = (uint32_t)__builtin_amdgcn_readfirstlane((int)sh.cand[tot - 1]);
            const bool open_here = has_open && (seg0 + (int)(cwl >> 3)) * kSeg + (int)(cwl & 7u) * kSub + kSub >= nb;
            if (!chain) {
                for (int wi = wv - 1; wi < nwin; wi += kResolveWaves - 1) {
                    const int wg = wbase + wi, buf = wg % kRing;
                    // this window's loads go out before the wait for its buffer
                    const StageIn cur = stage_load(sh, wi * kWinCand, tot, seg0, nb, tt, src, d, pool);
                    bool halt = false;
                    for (int spin = 0;; ++spin) {
                        halt = lds_load(&sh.stop) != 0;
                        if (halt || lds_load(&sh.consumed) >= wg - kRing + 1) break;
                        if (spin >= kSpinLimit) {
                            give_up();
                            halt = true;
                            break;
                        }
                        __builtin_amdgcn_s_sleep(1);
                    }
                    if (halt) break;
                    stage_window(sh, sh.win[buf], m, cur, wi * kWinCand, tot, seg0, b, n, nb, S, N, C_in, src, d,
                                 WT, carry, open_here && wi == nwin - 1, sh.kmax[buf]);
                    lds_store(&sh.ready[buf], wg + 1);
                }
            } else {
                for (int wi = 0; wi < nwin;) {
                    const int wg = wbase + wi, buf = wg % kRing;
                    bool late = false;
                    for (int spin = 0; lds_load(&sh.ready[buf]) != wg + 1; ++spin) {
                        if (spin >= kSpinLimit || lds_load(&sh.stop) != 0) {
                            if (spin >= kSpinLimit) give_up();
                            late = true;
                            break;
                        }
                        __builtin_amdgcn_s_sleep(1);
                    }
                    if (late) break;
                    // the run of windows wi, wi + 1, ... staged already (lane q
                    // looks at window wi + q), and the first of them whose
                    // largest key reaches the current deficit's key: the
                    // windows before it hold no crossing and are passed over
                    const int bq = (wg + lane) % kRing;
                    const bool rdy = lane < kRing && wi + lane < nwin && lds_load(&sh.ready[bq]) == wg + lane + 1;
                    const int nr = __builtin_ctzll(~__ballot(rdy));
                    const unsigned long long hit = __ballot(lane < nr && sh.kmax[bq] >= ch.K);
                    if (hit == 0ull) {
                        wi += nr;
                        lds_store(&sh.consumed, wg + nr);
                        continue;
                    }
                    wi += __builtin_ctzll(hit);
                    const int wh = wbase + wi, c0 = wi * kWinCand;
                    chain_window<PI>(sh, sh.win[wh % kRing], m, wh, c0, min(kWinCand, tot - c0) * kSub,
                                     open_here && wi == nwin - 1, seg0, nb, ch, st, si, sk);
                    ++wi;
                    lds_store(&sh.consumed, wh + 1);
                    if (ch.capped) {
                        lds_store(&sh.stop, 1);
                        break;
                    }
                }
            }
        }
        wbase += nwin;
        __syncthreads();                      // both waves are done with the chunk's list
        stop = __builtin_amdgcn_readfirstlane(lds_load(&sh.stop)) != 0;
    }
    if (!chain) return 0;
    flush_spikes(sh, m, ch.ns - ch.ns % kWave, ch.ns, st, si, sk);
    if (lane == 0) out_n[idx] = ch.ns;
    return ch.ns;
}

// Work-list driven: the per-sample lists of neurons built by the check pass
// are taken as one concatenated list, entry w by workgroup w mod gridDim.x.
// Status counts are added once per workgroup.
template <int PI>
__global__ __launch_bounds__(kWave * kResolveWaves) void k_resolve(
    const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src, const int32_t* __restrict__ ev_n, int B,
    int E_max, const float* __restrict__ WT, int C_in, int N, int E_pad, int S, Model m,
    const Decay* __restrict__ dec, const double2* __restrict__ carry, const uint32_t* __restrict__ mask,
    uint32_t pool_cap, const double2* __restrict__ pool, const uint32_t* __restrict__ pool_count,
    const uint32_t* __restrict__ work, const uint32_t* __restrict__ nwork, float* __restrict__ out_t,
    int32_t* __restrict__ out_n, float* __restrict__ out_i, int32_t* __restrict__ out_k, int32_t* __restrict__ status)
{
    __shared__ ResolveLds sh;
    const int lane = (int)threadIdx.x % kWave;
    if (blockIdx.x == gridDim.x - 1 && threadIdx.x >= blockDim.x - kWave) {
        // status words fixed once the check pass has run (the only writer of
        // these words in the call): events consumed, flagged sub-blocks,
        // sub-blocks past the pool's capacity
        unsigned long long ev = 0, fl = 0, fb = 0;
        for (int bb = lane; bb < B; bb += kWave) {
            ev += (unsigned long long)clamp_count(ev_n[bb], E_max);
            const uint32_t pc = pool_count[(size_t)bb * kCtr];
            fl += pc;
            fb += pc > pool_cap ? pc - pool_cap : 0u;
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            ev += __shfl_xor(ev, off, kWave);
            fl += __shfl_xor(fl, off, kWave);
            fb += __shfl_xor(fb, off, kWave);
        }
        if (lane == 0) {
            auto sat = [](unsigned long long x) { return (int32_t)(x > 0x7fffffffull ? 0x7fffffffull : x); };
            status[LIF_ST_EVENTS] = sat(ev);
            status[LIF_ST_CAND_BLOCKS] = sat(fl);
            status[LIF_ST_WALKED_BLOCKS] = sat(fl);
            status[LIF_ST_POOL_FALLBACK] = sat(fb);
        }
    }
    // spikes and capped neurons of this workgroup's neurons, added to the
    // status words once at its end
    unsigned long long spikes = 0;
    uint32_t capped = 0;
    // Both waves walk the list the same way.  Running sum of the list
    // lengths over groups of 64 samples (one load per lane, a wave prefix
    // sum): entry w of the concatenated lists belongs to the first sample
    // whose running sum exceeds w.
    int b0 = 0;               // first sample of the current group
    uint32_t base = 0;        // entries of the samples before the group
    uint32_t incl = 0;        // running sum up to and including sample b0 + lane
    auto load_group = [&]() {
        uint32_t c = b0 + lane < B ? nwork[(size_t)(b0 + lane) * kCtr] : 0u;
#pragma unroll
        for (int off = 1; off < kWave; off <<= 1) {
            const uint32_t v = (uint32_t)__shfl_up((int)c, off, kWave);
            if (lane >= off) c += v;
        }
        incl = base + c;
    };
    load_group();
    for (uint32_t w = blockIdx.x;; w += gridDim.x) {
        unsigned long long past = __ballot(b0 + lane < B && incl <= w);
        while (past == ~0ull) {              // w lies beyond the whole group
            base = (uint32_t)__shfl((int)incl, kWave - 1, kWave);
            b0 += kWave;
            if (b0 >= B) break;
            load_group();
            past = __ballot(b0 + lane < B && incl <= w);
        }
        const int l = __popcll(past);        // samples of the group whose entries end at or before w
        const int b = b0 + l;
        if (b0 >= B || l >= kWave || b >= B) break;
        const uint32_t before = l > 0 ? (uint32_t)__shfl((int)incl, l - 1, kWave) : base;
        const uint32_t bn = (uint32_t)__builtin_amdgcn_readfirstlane((int)work[(size_t)b * N + (w - before)]);
        const int ns = resolve_neuron<PI>(sh, (int)(bn / (uint32_t)N), (int)(bn % (uint32_t)N), ev_t, ev_src, ev_n,
                                      E_max, WT, C_in, N, E_pad, S, m, dec, carry, mask, pool_cap, pool, out_t, out_n,
                                      out_i, out_k, status);
        spikes += (unsigned long long)ns;
        capped += ns >= m.s_max ? 1u : 0u;
    }
    if (threadIdx.x == 0) {
        const int32_t sp = (int32_t)(spikes > 0x7fffffffull ? 0x7fffffffull : spikes);
        if (sp) {
            atomicAdd(&status[LIF_ST_SPIKES], sp);
            atomicAdd(&status[LIF_ST_ROOT_SOLVES], sp);
        }
        if (capped) {
            atomicAdd(&status[LIF_ST_CAPPED], (int32_t)capped);
            atomicOr(&status[LIF_ST_FLAGS], LIF_WARN_SPIKE_CAP);
        }
    }
}

// Status words of a sequential forward call, from what the pass wrote:
// spikes and capped neurons from the counts, events from the queue lengths.
// Each workgroup adds its sums with one atomic per word (one workgroup per
// kStatusPer counts); the status words start at zero (reset by k_prep).  The
// parallel path fills the same words inside its resolve pass.
constexpr int kStatusThreads = 1024;
constexpr int kStatusBatch = 8;
constexpr int kStatusPer = kStatusThreads * kStatusBatch;

__global__ __launch_bounds__(kStatusThreads) void k_status(const int32_t* __restrict__ ev_n, int B, int E_max, int N,
                                                           int s_max, const int32_t* __restrict__ out_n,
                                                           int32_t* __restrict__ status)
{
    __shared__ unsigned long long part[kStatusThreads / kWave][3];
    unsigned long long spikes = 0, capped = 0, events = 0;
    const size_t nn = (size_t)B * (size_t)N;
    for (size_t i0 = (size_t)blockIdx.x * kStatusPer + threadIdx.x; i0 < nn; i0 += (size_t)gridDim.x * kStatusPer) {
        int c[kStatusBatch];
#pragma unroll
        for (int u = 0; u < kStatusBatch; ++u) {
            const size_t i = i0 + (size_t)u * kStatusThreads;
            c[u] = i < nn ? out_n[i] : 0;
        }
#pragma unroll
        for (int u = 0; u < kStatusBatch; ++u) {
            spikes += (unsigned long long)c[u];
            capped += c[u] >= s_max ? 1u : 0u;
        }
    }
    if (blockIdx.x == 0) {
        for (int b = threadIdx.x; b < B; b += kStatusThreads)
            events += (unsigned long long)clamp_count(ev_n[b], E_max);
    }
    unsigned long long v[3] = {spikes, capped, events};
#pragma unroll
    for (int q = 0; q < 3; ++q) {
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) v[q] += __shfl_xor(v[q], off, kWave);
    }
    const int wave = (int)threadIdx.x / kWave;
    if (threadIdx.x % kWave == 0) {
#pragma unroll
        for (int q = 0; q < 3; ++q) part[wave][q] = v[q];
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long t[3] = {0, 0, 0};
        for (int w = 0; w < kStatusThreads / kWave; ++w)
            for (int q = 0; q < 3; ++q) t[q] += part[w][q];
        auto sat = [](unsigned long long x) { return (int32_t)(x > 0x7fffffffull ? 0x7fffffffull : x); };
        if (t[0]) {
            atomicAdd(&status[LIF_ST_SPIKES], sat(t[0]));
            atomicAdd(&status[LIF_ST_ROOT_SOLVES], sat(t[0]));
        }
        if (t[1]) {
            atomicAdd(&status[LIF_ST_CAPPED], sat(t[1]));
            atomicOr(&status[LIF_ST_FLAGS], LIF_WARN_SPIKE_CAP);
        }
        if (t[2]) atomicAdd(&status[LIF_ST_EVENTS], sat(t[2]));
    }
}

static unsigned status_blocks(int B, int N)
{
    const size_t nn = (size_t)B * (size_t)N;
    const size_t g = (nn + kStatusPer - 1) / kStatusPer;
    return (unsigned)(g < 1 ? 1 : (g > 64 ? 64 : g));
}

// Sequential baseline (Appendix E.3): one thread per (sample, neuron)
// consumes every event in order with the same interval test and root solve.
// The state (V, I) is the true one, so each interval starts with deficit 0;
// spikes inside it raise the deficit and the rest of the interval is
// re-tested.
// QUEUE: every neuron has its own queue (a layer with synaptic delays):
// ev_t holds the arrival times [B][N][E_max], q_k the sample's event index of
// each entry, and each thread computes its own decays (no shared table).
template <bool QUEUE>
__global__ __launch_bounds__(64) void k_sequential(const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src,
                                                   const int32_t* __restrict__ ev_n, const int32_t* __restrict__ q_k,
                                                   int B, int E_max, const float* __restrict__ WT, int C_in, int N,
                                                   Model m, int E_pad, const Decay* __restrict__ dec,
                                                   float* __restrict__ out_t, int32_t* __restrict__ out_n,
                                                   float* __restrict__ out_i, int32_t* __restrict__ out_k)
{
    const size_t idx_raw = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const bool live = idx_raw < (size_t)B * (size_t)N;
    const size_t idx = live ? idx_raw : 0;            // lanes past the end run neuron 0 and write nothing
    int b = (int)(idx / (size_t)N), n = (int)(idx % (size_t)N);
    int nb = clamp_count(ev_n[b], E_max);
    const float* tt = ev_t + (QUEUE ? idx : (size_t)b) * (size_t)E_max;
    const int32_t* src = ev_src + (size_t)b * E_max;
    const int32_t* qk = QUEUE ? q_k + idx * (size_t)E_max : nullptr;
    const Decay* d = QUEUE ? nullptr : dec + (size_t)b * E_pad;
    float* st = out_t + idx * (size_t)m.s_max;
    float* si = out_i ? out_i + idx * (size_t)m.s_max : nullptr;
    int32_t* sk = out_k ? out_k + idx * (size_t)m.s_max : nullptr;
    int ns = 0;
    bool capped = false;
    double V = 0.0, I = 0.0, t_prev = 0.0;
    for (int k = 0; k <= nb && !capped; ++k) {
        double L, A, C, Dd;
        if (k < nb) {
            const Decay e = QUEUE ? make_decay(m, tt, k) : d[k];
            A = e.A; C = e.C; Dd = e.D;
            L = (double)tt[k] - t_prev;
        } else {
            L = m.t_end - t_prev;                      // open interval after the last event
            if (!(L > 0.0)) break;
            if (isinf(L)) {
                A = 0.0; C = 0.0; Dd = 0.0;
            } else {
                A = exp(-L * m.inv_tm);
                Dd = exp(-L * m.inv_ts);
                C = unit_kernel(m, L, A);
            }
        }
        double V1 = A * V + C * I;
        // no-crossing screen V0 + max(I0 - th, 0) L / tm >= th_lo (screen_value)
        if (L > 0.0 && V + (I > m.th ? (I - m.th) * (L * m.inv_tm) : 0.0) >= m.th_lo) {
            IntervalMax im = interval_max(m, V, I, V1, L, A, Dd);
            double Dk = 0.0, lo = 0.0, ylo = 1.0, Flo = V - m.th;
            const double kI = m.kappa * I;
            while (Dk * im.a <= im.g) {
                const SpikeY sp = solve_spike_y(m, V - Dk + kI, kI, lo, ylo, Flo, im.hi, im.Fhi - Dk);
                const double u = -m.tm * log(sp.y);
                if (live) {
                    st[ns] = (float)(t_prev + u);
                    if (si) si[ns] = (float)(I * (sp.E2 * sp.y));
                    if (sk) sk[ns] = k;
                }
                ++ns;
                Dk += m.dth * sp.E1;
                lo = u;
                ylo = sp.y;
                Flo = -m.dth * sp.E1;
                if (ns >= m.s_max) { capped = true; break; }
            }
            V1 -= Dk * A;                               // true V at the end of the interval
        }
        V = V1;
        if (k < nb) {
            const int se = QUEUE ? min(max(qk[k], 0), nb - 1) : k;
            I = Dd * I + (double)WT[(size_t)clamp_src(src[se], C_in) * (size_t)N + n];
            t_prev = (double)tt[k];
        }
    }
    if (live) {
        out_n[idx] = ns;
        for (int s = ns; s < m.s_max; ++s) {
            st[s] = INFINITY;
            if (si) si[s] = 0.0f;
            if (sk) sk[s] = 0;
        }
    }
}

__global__ void k_status_zero(int32_t* __restrict__ status)
{
    if (threadIdx.x < LIF_STATUS_WORDS) status[threadIdx.x] = 0;
}

int launch_sequential_queue(const float* q_t, const int32_t* q_k, const int32_t* ev_src, const int32_t* ev_n, int B,
                            int E_max, const float* WT, int C_in, int N, const Model& m, float* out_t, int32_t* out_n,
                            float* out_i, int32_t* out_k, int32_t* status, hipStream_t stream)
{
    const size_t nn = (size_t)B * N;
    TIMED_LAUNCH("status_zero", k_status_zero, dim3(1), dim3(kWave), 0, stream, status);
    if (nn)
        TIMED_LAUNCH("sequential", k_sequential<true>, dim3((unsigned)((nn + 63) / 64)), dim3(64), 0, stream, q_t,
                     ev_src, ev_n, q_k, B, E_max, WT, C_in, N, m, 0, nullptr, out_t, out_n, out_i, out_k);
    TIMED_LAUNCH("status", k_status, dim3(status_blocks(B, N)), dim3(kStatusThreads), 0, stream, ev_n, B, E_max, N,
                 m.s_max, out_n, status);
    return check_launch();
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
FwdLayout fwd_layout(int B, int E_max, int N, int pool_cap)
{
    FwdLayout L{};
    L.S = (E_max + kSeg - 1) / kSeg;
    L.E_pad = L.S * kSeg;
    size_t off = 0;
    auto take = [&](size_t bytes) { size_t o = off; off += (bytes + 255) & ~(size_t)255; return o; };
    const size_t BS = (size_t)B * L.S;
    L.dec = take((size_t)B * L.E_pad * sizeof(Decay));
    L.segm = take(BS * sizeof(double2));
    // segment aggregates, overwritten in place by the carried states
    L.carry = take(BS * N * sizeof(double2));
    L.mask = take(BS * N * sizeof(uint32_t));
    // per sample: pool use, work-list length
    L.n_counters = 2 * (size_t)B * kCtr;
    L.counters = take(L.n_counters * sizeof(uint32_t));
    L.listed = take((size_t)B * N * sizeof(uint32_t));
    L.work = take((size_t)B * N * sizeof(uint32_t));
    // Pool of entering states: one 16-byte entry per flagged (sub-block,
    // neuron), in per-sample slices sized at a quarter of the dense bound
    // (every sub-block of every neuron flagged), at least 4096 entries (the
    // dense bound when smaller), and at most 1 GiB in all unless that leaves
    // fewer than 4096 per sample.  A full slice only sends the excess
    // sub-blocks through a slower rebuild from the segment's carried state,
    // with identical results.  lif_params.pool_cap >= 0 sets the slice size.
    const size_t dense = (size_t)L.S * kSubPerSeg * N;
    size_t cap = dense / 4 > 4096 ? dense / 4 : (dense < 4096 ? dense : 4096);
    const size_t budget = (size_t)1 << 30;
    if (B > 0 && (size_t)B * cap * sizeof(double2) > budget) {
        const size_t fit = budget / ((size_t)B * sizeof(double2));
        const size_t floor_ = dense < 4096 ? dense : 4096;
        cap = fit > floor_ ? fit : floor_;
    }
    if (pool_cap >= 0) cap = (size_t)pool_cap;
    if (B > 0 && (size_t)B * cap > 0xfffffff0ull) cap = 0xfffffff0ull / (size_t)B;   // slot indices are 32-bit
    L.pool_cap = cap;
    const size_t recs = (size_t)B * cap;
    L.pool = take((recs > 0 ? recs : 1) * sizeof(double2));   // at least one entry (a safe load address)
    L.total = off + 256;
    return L;
}

// Neurons per lane of the segment walks: NPL-wide weight loads need W^T rows
// of a multiple of NPL floats and an aligned base.
static int pick_npl(const float* WT, int N)
{
    const uintptr_t a = (uintptr_t)WT;
    if (N % 4 == 0 && a % 16 == 0) return 4;
    if (N % 2 == 0 && a % 8 == 0) return 2;
    return 1;
}

struct FwdPtrs {
    Decay* dec;
    double2 *segm, *carry;
    uint32_t* mask;
    uint32_t *counters, *pool_count, *nwork, *listed, *work;
    double2* pool;
};

template <int NPL>
static void launch_walks(const FwdLayout& L, const FwdPtrs& P, const float* ev_t, const int32_t* ev_src,
                         const int32_t* ev_n, int B, int E_max, const float* WT, int C_in, int N, const Model& m,
                         int32_t* status, bool validate, int32_t* out_n, float* out_t, float* out_i, int32_t* out_k,
                         hipStream_t stream, bool check = true)
{
    const int tiles = (N + kWave * NPL - 1) / (kWave * NPL);
    const size_t items = (size_t)B * L.S * tiles;
    const unsigned blocks = (unsigned)((items + kWalkWaves - 1) / kWalkWaves);
    // the aggregate pass also computes the decays and resets the counters and
    // status words (validation flags are ORed in after it)
    TIMED_LAUNCH("aggregate", k_aggregate<NPL>, dim3(blocks), dim3(kWave * kWalkWaves), 0, stream,
                 ev_t, ev_src, ev_n, E_max, L.E_pad, WT, C_in, N, tiles, L.S, (int)items, m, P.dec, P.segm,
                 P.carry, status, P.counters, L.n_counters, P.listed, (size_t)B * N, out_n, out_t, out_i, out_k,
                 out_t ? (size_t)B * N * (size_t)m.s_max : (size_t)0);
    if (validate)
        TIMED_LAUNCH("validate", k_validate, dim3((unsigned)(((size_t)B * E_max + 255) / 256)), dim3(256), 0,
                     stream, ev_t, ev_src, ev_n, B, E_max, C_in, status);
    const int ctiles = (N + kWave - 1) / kWave;
    TIMED_LAUNCH("carry", k_carry, dim3((unsigned)((size_t)B * ctiles)), dim3(kWave * kCarryWaves), 0, stream,
                 ev_n, B, E_max, N, ctiles, L.S, P.segm, P.carry, P.carry);
    if (!check) return;
    // The check pass takes one neuron per lane whatever NPL the aggregate
    // uses: its screen and pool state make wider lanes cost occupancy
    // (about 200 VGPRs at four neurons per lane against under 80 at one).
    const int ctl = (N + kWave - 1) / kWave;
    const size_t citems = (size_t)B * L.S * ctl;
    const unsigned cblocks = (unsigned)((citems + kWalkWaves - 1) / kWalkWaves);
    TIMED_LAUNCH("check", k_check, dim3(cblocks), dim3(kWave * kWalkWaves), 0, stream,
                 ev_t, ev_src, ev_n, E_max, L.E_pad, WT, C_in, N, ctl, L.S, (int)citems, m, P.dec, P.carry, P.mask,
                 P.pool, P.pool_count, (uint32_t)L.pool_cap, P.listed, P.work, P.nwork);
}

int forward_impl(bool sequential, const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                 const float* WT, int C_in, int N, const lif_params* p, float* out_t, int32_t* out_n,
                 float* out_i, int32_t* out_k, int32_t* status, void* ws, size_t ws_bytes, hipStream_t stream)
{
    int rc = validate_forward_args(ev_t, ev_src, ev_n, B, E_max, WT, C_in, N, p, out_t, out_n, status);
    if (rc) return rc;
    if (!ws) return LIF_ERR_ARG;
    FwdLayout L = fwd_layout(B, E_max, N, p->pool_cap);
    if (ws_bytes < L.total) return LIF_ERR_WORKSPACE;
    Model m = make_model(*p);
    char* base = (char*)(((uintptr_t)ws + 255) & ~(uintptr_t)255);
    FwdPtrs P;
    P.dec = (Decay*)(base + L.dec);
    P.segm = (double2*)(base + L.segm);
    P.carry = (double2*)(base + L.carry);
    P.mask = (uint32_t*)(base + L.mask);
    P.counters = (uint32_t*)(base + L.counters);
    P.pool_count = P.counters;
    P.nwork = P.counters + (size_t)B * kCtr;
    P.listed = (uint32_t*)(base + L.listed);
    P.work = (uint32_t*)(base + L.work);
    P.pool = (double2*)(base + L.pool);

    const size_t nev = (size_t)B * L.E_pad;
    const size_t nn = (size_t)B * N;
    const size_t items_max = (size_t)B * L.S * ((N + kWave - 1) / kWave);
    if (items_max > 0x7fffffff || nn > 0xffffffffull) return LIF_ERR_SIZE;
    // mask words hold a per-sample pool offset in 28 bits
    if ((size_t)L.S * kSubPerSeg * N >= ((size_t)1 << (32 - kMaskBits))) return LIF_ERR_SIZE;
    const size_t n_out = nn * (size_t)p->s_max;
    const bool validate = (p->flags & LIF_VALIDATE) && (size_t)B * E_max;
    if (sequential || items_max == 0) {
        // decays and resets in their own pass (the parallel path folds them
        // into the aggregate and carry passes)
        size_t work_items = nev > n_out ? nev : n_out;
        size_t blocks = (work_items + 255) / 256;
        if (blocks > 2048) blocks = 2048;
        if (blocks < 1) blocks = 1;
        TIMED_LAUNCH("prep", k_prep, dim3((unsigned)blocks), dim3(256), 0, stream,
                     ev_t, ev_n, B, E_max, L.E_pad, L.S, m, P.dec, sequential ? nullptr : P.segm, status, P.counters,
                     L.n_counters, out_n, sequential ? nullptr : P.listed, nn, sequential ? nullptr : out_t, out_i,
                     out_k, n_out);
        if (validate)
            TIMED_LAUNCH("validate", k_validate, dim3((unsigned)(((size_t)B * E_max + 255) / 256)), dim3(256), 0,
                         stream, ev_t, ev_src, ev_n, B, E_max, C_in, status);
    }
    if (sequential) {
        if (nn)
            TIMED_LAUNCH("sequential", k_sequential<false>, dim3((unsigned)((nn + 63) / 64)), dim3(64), 0, stream,
                         ev_t, ev_src, ev_n, nullptr, B, E_max, WT, C_in, N, m, L.E_pad, P.dec, out_t, out_n, out_i,
                         out_k);
        TIMED_LAUNCH("status", k_status, dim3(status_blocks(B, N)), dim3(kStatusThreads), 0, stream, ev_n, B, E_max, N, m.s_max, out_n,
                     status);
        return check_launch();
    }
    if (items_max == 0) return check_launch();
    switch (pick_npl(WT, N)) {
    case 4: launch_walks<4>(L, P, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N, m, status, validate, out_n, out_t, out_i,
                            out_k, stream); break;
    case 2: launch_walks<2>(L, P, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N, m, status, validate, out_n, out_t, out_i,
                            out_k, stream); break;
    default: launch_walks<1>(L, P, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N, m, status, validate, out_n, out_t,
                             out_i, out_k, stream); break;
    }
    // Four-wave workgroups (a chain wave and three staging waves) over the
    // concatenated per-sample lists, as many as are resident at once; one
    // kernel per spike-time solver (the polynomial degree)
    const unsigned rgrid = (unsigned)(nn < 1024 ? nn : 1024);
    auto resolve = [&](auto kern) {
        TIMED_LAUNCH("resolve", kern, dim3(rgrid), dim3(kWave * kResolveWaves), 0, stream,
                     ev_t, ev_src, ev_n, B, E_max, WT, C_in, N, L.E_pad, L.S, m, P.dec, P.carry, P.mask,
                     (uint32_t)L.pool_cap, P.pool, P.pool_count, P.work, P.nwork, out_t, out_n, out_i, out_k,
                     status);
    };
    switch (m.p_int) {
    case 1: resolve(k_resolve<1>); break;
    case 2: resolve(k_resolve<2>); break;
    case 3: resolve(k_resolve<3>); break;
    case 4: resolve(k_resolve<4>); break;
    default: resolve(k_resolve<0>); break;
    }
    return check_launch();
}

}  // namespace lif

extern "C" size_t lif_layer_forward_workspace_size(int B, int E_max, int C_in, int N_out, const lif_params* p)
{
    (void)C_in;
    if (B < 0 || E_max < 0 || N_out < 1 || !p) return 0;
    return lif::fwd_layout(B, E_max, N_out, p->pool_cap).total;
}

extern "C" int lif_layer_forward(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                                 const float* WT, int C_in, int N_out, const lif_params* p, float* out_t,
                                 int32_t* out_n, float* out_i, int32_t* out_k, int32_t* status, void* ws,
                                 size_t ws_bytes, lif_stream_t stream)
{
    return lif::forward_impl(false, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, p, out_t, out_n, out_i, out_k,
                             status, ws, ws_bytes, (hipStream_t)stream);
}

extern "C" int lif_layer_forward_sequential(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B,
                                            int E_max, const float* WT, int C_in, int N_out, const lif_params* p,
                                            float* out_t, int32_t* out_n, float* out_i, int32_t* out_k,
                                            int32_t* status, void* ws, size_t ws_bytes, lif_stream_t stream)
{
    return lif::forward_impl(true, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, p, out_t, out_n, out_i, out_k,
                             status, ws, ws_bytes, (hipStream_t)stream);
}

namespace lif {

// ---------------------------------------------------------------------------
// Spike-count regularisers (App. E.1, Eq. loss): for every (sample, neuron)
// and every input interval j (between events j - 1 and j, and the open one
// after the last event up to t_end), the largest V of the interval's
// trajectory from its true start state (resets of earlier intervals
// applied, none inside it), split into the intervals that hold a spike
// (out_k = j) and the silent ones.  The no-reset state comes from the
// forward's segment scan (k_aggregate, k_carry); the resets enter as the
// decaying deficit (V_th - V_reset) e^{-(t - t_s)/tm} of each earlier spike.
// ---------------------------------------------------------------------------


// Per (sample, segment, 64 neurons): the segment's intervals (and the open
// one in the sample's last segment); per lane the sums of the hinge terms
// and the interval counts, part = (sum under, silent count, sum over,
// spiking count); with rec, the per-interval records and, per (sample,
// segment, neuron), the sums over the segment's active intervals of the
// decays from the segment's start (the input event before it) to the
// interval's argmax, local = (under: e^{-./tm}, e^{-./ts}; over: the same).
__global__ __launch_bounds__(kWave * kWalkWaves) void k_reg_walk(
    const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src, const int32_t* __restrict__ ev_n, int E_max,
    int E_pad, const float* __restrict__ WT, int C_in, int N, int tiles, int S, int items, Model m,
    const Decay* __restrict__ dec, const double2* __restrict__ carry, const float* __restrict__ out_t,
    const int32_t* __restrict__ out_n, const int32_t* __restrict__ out_k, double4* __restrict__ part,
    float2* __restrict__ rec, double4* __restrict__ local)
{
    __shared__ double2 s_ad[kWalkWaves][kSeg];
    __shared__ float s_t[kWalkWaves][kSeg + 1];
    WalkCoords c;
    if (!walk_coords<1>(items, tiles, S, ev_n, E_max, N, c)) return;
    const int lane = c.lane, wv = (int)threadIdx.x / kWave;
    const int n = c.n0;
    double2* lad = s_ad[wv];
    float* lt = s_t[wv];
    const float* tt = ev_t + (size_t)c.b * E_max;
    const Stage st = stage_segment(c, ev_src + (size_t)c.b * E_max + c.k0, dec + (size_t)c.b * E_pad + c.k0, WT,
                                   C_in, N, lad, nullptr, nullptr);
    // lt[e] = start of interval k0 + e (the time of event k0 + e - 1, or 0)
#pragma unroll
    for (int h = 0; h < kSrcRegs; ++h) {
        const int e = h * kWave + lane;
        if (e < c.cnt) lt[e + 1] = tt[c.k0 + e];
    }
    if (lane == 0) lt[0] = c.k0 > 0 ? tt[c.k0 - 1] : 0.0f;
    wave_lds_sync();
    const double2 cs = carry[((size_t)c.b * S + c.seg) * N + n];
    double U = cs.x, J = cs.y;
    // the neuron's spikes: the deficit at the segment's start from those of
    // earlier intervals, then the ones inside taken in order
    const size_t base = ((size_t)c.b * N + n) * (size_t)m.s_max;
    const float* ts = out_t + base;
    const int32_t* ks = out_k + base;
    const int ns = c.live ? min(out_n[(size_t)c.b * N + n], m.s_max) : 0;
    const double t_start = (double)lt[0];
    double Dft = 0.0;
    int sp = 0;
    while (sp < ns && ks[sp] < c.k0) {
        Dft += m.dth * exp(-(t_start - (double)ts[sp]) * m.inv_tm);
        ++sp;
    }
    double su = 0.0, so = 0.0;
    int nsil = 0, nspk = 0;
    float2* rb = rec ? rec + (size_t)c.b * (E_max + 1) * N + n : nullptr;
    double cdm = 1.0, cds = 1.0;                 // decays from the segment's start to the interval's start
    double4 loc = make_double4(0.0, 0.0, 0.0, 0.0);
    auto take = [&](int j, double L, double A, double Dd, double t1) {
        const double V0 = v_of(m, U, J) - Dft;
        const RegArg ra = reg_vmax_arg(m, V0, J, L, A, Dd);
        const double vmax = ra.vmax;
        const bool spiked = sp < ns && ks[sp] == j;
        if (spiked) {
            so += fmax(vmax - m.th, 0.0);
            ++nspk;
        } else {
            su += fmax(m.th - vmax, 0.0);
            ++nsil;
        }
        if (rb && c.live) {
            const float sgn = spiked ? (vmax > m.th ? -1.0f : 0.0f) : (vmax < m.th ? 1.0f : 0.0f);
            if (ra.at_start)
                rb[(size_t)j * N] = make_record(sgn, kRecStart, 1.0, 1.0, j > 0 ? (J - V0) * m.inv_tm : 0.0);
            else if (ra.at_end && j < c.nb)
                rb[(size_t)j * N] = make_record(sgn, kRecEnd, A, Dd, (J * Dd - ra.vmax) * m.inv_tm);
            else                                 // inside, or the end t_end of the open interval
                rb[(size_t)j * N] = make_record(sgn, kRecInside, ra.em, ra.es, 0.0);
            if (sgn > 0.0f) {
                loc.x = fma(cdm, ra.em, loc.x);
                loc.y = fma(cds, ra.es, loc.y);
            } else if (sgn < 0.0f) {
                loc.z = fma(cdm, ra.em, loc.z);
                loc.w = fma(cds, ra.es, loc.w);
            }
            cdm *= A;
            cds *= Dd;
        }
        // the deficit at the interval's end, with the spikes inside it
        Dft *= A;
        while (sp < ns && ks[sp] == j) {
            Dft += m.dth * exp(-(t1 - (double)ts[sp]) * m.inv_tm);
            ++sp;
        }
    };
    const int ng = (c.cnt + kGrp - 1) / kGrp;
    float wa[kGrp][1], wb[kGrp][1];
    load_grp<1>(st, 0, wa);
    auto group = [&](int g, const float (&w)[kGrp][1]) {
#pragma unroll
        for (int jj = 0; jj < kGrp; ++jj) {
            const int e = g * kGrp + jj;
            if (e >= c.cnt) break;
            const double2 ad = lad[e];
            const double t0 = (double)lt[e], t1 = (double)lt[e + 1];
            take(c.k0 + e, t1 - t0, ad.x, ad.y, t1);
            step1(ad, w[jj][0], U, J);
        }
    };
    for (int g = 0; g < ng; g += 2) {
        if (g + 1 < ng) load_grp<1>(st, (g + 1) * kGrp, wb);
        group(g, wa);
        if (g + 1 >= ng) break;
        if (g + 2 < ng) load_grp<1>(st, (g + 2) * kGrp, wa);
        group(g + 1, wb);
    }
    if (c.k0 + c.cnt == c.nb) {
        // the open interval after the sample's last event, up to t_end
        const double t0 = (double)lt[c.cnt];
        const double L = m.t_end - t0;
        const double A = isinf(L) ? 0.0 : exp(-L * m.inv_tm), Dd = isinf(L) ? 0.0 : exp(-L * m.inv_ts);
        take(c.nb, L, A, Dd, m.t_end);
    }
    if (c.live) part[((size_t)c.b * S + c.seg) * N + n] = make_double4(su, (double)nsil, so, (double)nspk);
    if (local && c.live) local[((size_t)c.b * S + c.seg) * N + n] = loc;
}

// Per (sample, neuron): the sums over the segments in order, then the means
// over the silent and the spiking intervals (0 for an empty set).
__global__ __launch_bounds__(256) void k_reg_reduce(const double4* __restrict__ part, const int32_t* __restrict__ ev_n,
                                                    int B, int E_max, int N, int S, double th, double* __restrict__ ub,
                                                    double* __restrict__ ob, float* __restrict__ under,
                                                    float* __restrict__ over, double2* __restrict__ counts)
{
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (size_t)B * N) return;
    const int b = (int)(i / (size_t)N), n = (int)(i % (size_t)N);
    const int nb = clamp_count(ev_n[b], E_max);
    const int Sb = (nb + kSeg - 1) / kSeg;
    double su = 0.0, nsil = 0.0, so = 0.0, nspk = 0.0;
    for (int s = 0; s < Sb; ++s) {
        const double4 p = part[((size_t)b * S + s) * N + n];
        su += p.x;
        nsil += p.y;
        so += p.z;
        nspk += p.w;
    }
    if (Sb == 0) {             // no event: the one interval [0, t_end) at rest (V_max = 0)
        su = th;
        nsil = 1.0;
    }
    const double u = nsil > 0.0 ? su / nsil : 0.0;
    const double o = nspk > 0.0 ? so / nspk : 0.0;
    ub[i] = u;
    ob[i] = o;
    if (under) under[i] = (float)u;
    if (over) over[i] = (float)o;
    if (counts) counts[i] = make_double2(nsil, nspk);
}

// The two loss terms (one workgroup): per neuron the batch means and the
// gates of the mean spike count against the target, then the means over the
// neurons, each sum in a fixed order.
constexpr int kRegThreads = 256;

__global__ __launch_bounds__(kRegThreads) void k_reg_loss(const double* __restrict__ ub, const double* __restrict__ ob,
                                                          const int32_t* __restrict__ out_n, int B, int N, int s_max,
                                                          double c_target, float* __restrict__ loss,
                                                          double2* __restrict__ gates)
{
    __shared__ double s_reg[kRegThreads], s_over[kRegThreads];
    double lr = 0.0, lo = 0.0;
    for (int n = threadIdx.x; n < N; n += kRegThreads) {
        double cb = 0.0, mu = 0.0, mo = 0.0, ov = 0.0;
        for (int b = 0; b < B; ++b) {
            const size_t i = (size_t)b * N + n;
            const double cnt = (double)min(out_n[i], s_max);
            cb += cnt;
            mu += ub[i];
            mo += ob[i];
            ov += fmax(cnt / c_target - 1.0, 0.0) * ob[i];
        }
        cb /= (double)B;
        const double gu = fmax(1.0 - cb / c_target, 0.0), go = fmax(cb / c_target - 1.0, 0.0);
        lr += gu * (mu / (double)B) + go * (mo / (double)B);
        lo += ov;
        if (gates) gates[n] = make_double2(gu, go);
    }
    s_reg[threadIdx.x] = lr;
    s_over[threadIdx.x] = lo;
    __syncthreads();
    for (int off = kRegThreads / 2; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off) {
            s_reg[threadIdx.x] += s_reg[threadIdx.x + off];
            s_over[threadIdx.x] += s_over[threadIdx.x + off];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0 && loss) {
        loss[0] = (float)(s_reg[0] / (double)N);
        loss[1] = (float)(s_over[0] / (double)N);
    }
}

void launch_reg_loss(const double* ub, const double* ob, const int32_t* out_n, int B, int N, int s_max,
                     double c_target, float* loss, double2* gates, hipStream_t stream)
{
    TIMED_LAUNCH("reg_loss", k_reg_loss, dim3(1), dim3(kRegThreads), 0, stream, ub, ob, out_n, B, N, s_max, c_target,
                 loss, gates);
}

struct RegLayout {
    FwdLayout f;
    size_t part, ub, ob, status, total;
};

static RegLayout reg_layout(int B, int E_max, int N)
{
    RegLayout R;
    R.f = fwd_layout(B, E_max, N, 0);
    size_t off = R.f.total;
    auto take = [&](size_t bytes) { size_t o = off; off += (bytes + 255) & ~(size_t)255; return o; };
    R.part = take((size_t)B * R.f.S * N * sizeof(double4));
    R.ub = take((size_t)B * N * sizeof(double));
    R.ob = take((size_t)B * N * sizeof(double));
    R.status = take(LIF_STATUS_WORDS * sizeof(int32_t));
    R.total = off + 256;
    return R;
}

}  // namespace lif

extern "C" size_t lif_spike_count_reg_workspace_size(int B, int E_max, int C_in, int N_out)
{
    (void)C_in;
    if (B < 0 || E_max < 0 || N_out < 1) return 0;
    return lif::reg_layout(B, E_max, N_out).total;
}

extern "C" int lif_spike_count_reg(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                                   const float* WT, int C_in, int N_out, const lif_params* p, const float* out_t,
                                   const int32_t* out_n, const int32_t* out_k, double c_target, float* loss,
                                   float* under, float* over, void* ws, size_t ws_bytes, lif_stream_t stream_)
{
    using namespace lif;
    int rc = validate_forward_args(ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, p, out_t, out_n, out_n);
    if (rc) return rc;
    if (!out_k || !loss || !ws || !(c_target > 0.0) || !isfinite(c_target)) return LIF_ERR_ARG;
    const RegLayout R = reg_layout(B, E_max, N_out);
    if (ws_bytes < R.total) return LIF_ERR_WORKSPACE;
    const size_t items_max = (size_t)B * R.f.S * ((N_out + kWave - 1) / kWave);
    if (items_max > 0x7fffffff) return LIF_ERR_SIZE;
    hipStream_t stream = (hipStream_t)stream_;
    const Model m = make_model(*p);
    char* base = (char*)(((uintptr_t)ws + 255) & ~(uintptr_t)255);
    FwdPtrs P{};
    P.dec = (Decay*)(base + R.f.dec);
    P.segm = (double2*)(base + R.f.segm);
    P.carry = (double2*)(base + R.f.carry);
    P.mask = (uint32_t*)(base + R.f.mask);
    P.counters = (uint32_t*)(base + R.f.counters);
    P.pool_count = P.counters;
    P.nwork = P.counters + (size_t)B * kCtr;
    P.listed = (uint32_t*)(base + R.f.listed);
    P.work = (uint32_t*)(base + R.f.work);
    P.pool = (double2*)(base + R.f.pool);
    double4* part = (double4*)(base + R.part);
    double* ub = (double*)(base + R.ub);
    double* ob = (double*)(base + R.ob);
    int32_t* st = (int32_t*)(base + R.status);
    const size_t nn = (size_t)B * N_out;
    if (items_max > 0) {
        // the no-reset state entering every segment (the forward's scan)
        switch (pick_npl(WT, N_out)) {
        case 4: launch_walks<4>(R.f, P, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, m, st, false, nullptr, nullptr,
                                nullptr, nullptr, stream, false); break;
        case 2: launch_walks<2>(R.f, P, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, m, st, false, nullptr, nullptr,
                                nullptr, nullptr, stream, false); break;
        default: launch_walks<1>(R.f, P, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, m, st, false, nullptr,
                                 nullptr, nullptr, nullptr, stream, false); break;
        }
        const int tl = (N_out + kWave - 1) / kWave;
        const size_t it = (size_t)B * R.f.S * tl;
        TIMED_LAUNCH("reg_walk", k_reg_walk, dim3((unsigned)((it + kWalkWaves - 1) / kWalkWaves)),
                     dim3(kWave * kWalkWaves), 0, stream, ev_t, ev_src, ev_n, E_max, R.f.E_pad, WT, C_in, N_out, tl,
                     R.f.S, (int)it, m, P.dec, P.carry, out_t, out_n, out_k, part, nullptr, nullptr);
    }
    if (nn)
        TIMED_LAUNCH("reg_reduce", k_reg_reduce, dim3((unsigned)((nn + 255) / 256)), dim3(256), 0, stream, part, ev_n,
                     B, E_max, N_out, R.f.S, m.th, ub, ob, under, over, nullptr);
    if (B > 0)
        TIMED_LAUNCH("reg_loss", k_reg_loss, dim3(1), dim3(kRegThreads), 0, stream, ub, ob, out_n, B, N_out, m.s_max,
                     c_target, loss, nullptr);
    return check_launch();
}

// ---------------------------------------------------------------------------
// Gradient of lam_reg L_reg + lam_over L_over (App. E.1, Eq. loss), the gates
// held constant (functions of the spike counts).  Each V_max is the value of
// its interval's trajectory at the argmax tau_j = t_{j-1} + u_j:
//   V(tau) = sum_{k < j} w_k K(tau - t_k) - (V_th - V_reset) sum_{s: out_k < j} e^{-(tau - t_s)/tm},
// so with mu_j = dL/dV_max of interval j (G_u for an active under-firing
// interval, G_o for an active over-firing one, 0 otherwise) and
//   P_k = sum_{j > k} mu_j e^{-(tau_j - t_k)/tm}    (Q_k the same with ts)
// every input event k collects
//   dL/dw_{i, src_k} += kappa (P_k - Q_k),   dL/dt_k += w kappa (P_k/tm - Q_k/ts)
// (the adjoint sums of the layer's backward pass with a pseudo-spike at
// each interval's argmax), an argmax at an interval end that is an input
// time adds mu_j V'(tau_j) to that time's gradient, and spike s collects the
// upstream spike-time gradient -((V_th - V_reset)/tm) P_{out_k} e^{-(t_{out_k} - t_s)/tm},
// which the layer's backward pass carries to W and the input times.
// P obeys P_{k-1} = A_k P_k + mu_k e^{-u_k/tm} (A_k the decay into event k),
// a reverse affine scan: per segment the sums over its own intervals (taken
// by k_reg_walk on its forward walk, split by hinge so that the multipliers,
// known only once the whole batch is walked, enter later), a reverse carry
// over segments (k_regg_carry), and the walk back with the carry
// (k_regg_walk).  dL/dW is added as 64-bit fixed-point integers (order
// free); dL/dt per neuron tile, the tiles added in order.
// ---------------------------------------------------------------------------
namespace lif {


// Per (sample, neuron): G_u = -lam_reg gu / (N B nsil), G_o = (lam_reg go /
// (N B) + lam_over gi / N) / nspk with gi = ReLU(c / c_target - 1) of its
// spike count c, and |G_u| nsil + |G_o| nspk, a bound of its sums P and Q.
__global__ __launch_bounds__(256) void k_regg_coef(const double2* __restrict__ counts,
                                                   const double2* __restrict__ gates,
                                                   const int32_t* __restrict__ out_n, int B, int N, int s_max,
                                                   double c_target, double lam_reg, double lam_over,
                                                   double2* __restrict__ coef, double* __restrict__ musum,
                                                   long long* __restrict__ gw, size_t nW)
{
    const size_t gtid = (size_t)blockIdx.x * blockDim.x + threadIdx.x, gs = (size_t)gridDim.x * blockDim.x;
    for (size_t x = gtid; x < nW; x += gs) gw[x] = 0;
    const size_t nn = (size_t)B * N;
    for (size_t i = gtid; i < nn; i += gs) {
        const int n = (int)(i % (size_t)N);
        const double2 cnt = counts[i], g = gates[n];
        const double c = (double)min(out_n[i], s_max);
        const double gi = fmax(c / c_target - 1.0, 0.0);
        const double Gu = cnt.x > 0.0 ? -lam_reg * g.x / ((double)N * B) / cnt.x : 0.0;
        const double Go = cnt.y > 0.0 ? (lam_reg * g.y / ((double)N * B) + lam_over * gi / (double)N) / cnt.y : 0.0;
        coef[i] = make_double2(Gu, Go);
        musum[i] = fabs(Gu) * cnt.x + fabs(Go) * cnt.y;
    }
}

void launch_regg_coef(const double2* counts, const double2* gates, const int32_t* out_n, int B, int N, int s_max,
                      double c_target, double lam_reg, double lam_over, double2* coef, double* musum,
                      hipStream_t stream)
{
    const size_t nn = (size_t)B * N;
    size_t blocks = (nn + 255) / 256;
    blocks = blocks < 1 ? 1 : (blocks > 2048 ? 2048 : blocks);
    TIMED_LAUNCH("regg_coef", k_regg_coef, dim3((unsigned)blocks), dim3(256), 0, stream, counts, gates, out_n, B, N,
                 s_max, c_target, lam_reg, lam_over, coef, musum, (long long*)nullptr, (size_t)0);
}

// Fixed-point scale of dL/dW (one workgroup): a contribution is at most
// 2 kappa M (M = the largest bound of k_regg_coef; the float32 decays of the
// records add far less than the bit of headroom), an element sums at most
// one per event of the batch: scale = 2^(61 - ceil(log2(2 kappa M events))).
__global__ __launch_bounds__(kRegThreads) void k_regg_scale(const double* __restrict__ musum, size_t nn,
                                                            const int32_t* __restrict__ ev_n, int B, int E_max,
                                                            double kappa, double* __restrict__ scale)
{
    __shared__ double s_max[kRegThreads], s_ev[kRegThreads];
    double mx = 0.0, ev = 0.0;
    for (size_t i = threadIdx.x; i < nn; i += kRegThreads) mx = fmax(mx, musum[i]);
    for (int b = threadIdx.x; b < B; b += kRegThreads) ev += (double)clamp_count(ev_n[b], E_max);
    s_max[threadIdx.x] = mx;
    s_ev[threadIdx.x] = ev;
    __syncthreads();
    for (int off = kRegThreads / 2; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off) {
            s_max[threadIdx.x] = fmax(s_max[threadIdx.x], s_max[threadIdx.x + off]);
            s_ev[threadIdx.x] += s_ev[threadIdx.x + off];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const double bound = 2.0 * kappa * s_max[0] * fmax(s_ev[0], 1.0);
        int ex = 0;
        if (bound > 0.0 && isfinite(bound)) frexp(bound, &ex);
        scale[0] = ldexp(1.0, 61 - ex);
    }
}

// Per (sample, 64 neurons): the reverse carry over segments.  F(seg) =
// (P, Q) at the input event before segment seg = its own part (local with the
// neuron's G) plus the later segments' F decayed over the segment (its
// composed decays segm); cin[seg] = F(seg + 1) = (P, Q) at the segment's last
// event, 0 for the last segment (its walk adds the open interval itself).
__global__ __launch_bounds__(kWave) void k_regg_carry(const int32_t* __restrict__ ev_n, int E_max, int N, int S,
                                                      const double2* __restrict__ segm,
                                                      const double4* __restrict__ local,
                                                      const double2* __restrict__ coef, double2* __restrict__ cin)
{
    const int b = blockIdx.y, n = blockIdx.x * kWave + (int)threadIdx.x;
    if (n >= N) return;
    const int nb = clamp_count(ev_n[b], E_max);
    const int Sb = (nb + kSeg - 1) / kSeg;
    const double2 G = coef[(size_t)b * N + n];
    double Fm = 0.0, Fs = 0.0;
#pragma unroll 8
    for (int seg = Sb - 1; seg >= 0; --seg) {
        const size_t at = ((size_t)b * S + seg) * N + n;
        const double4 L = local[at];
        const double2 f = segm[(size_t)b * S + seg];
        cin[at] = make_double2(Fm, Fs);
        Fm = fma(f.x, Fm, fma(G.x, L.x, G.y * L.z));
        Fs = fma(f.y, Fs, fma(G.x, L.y, G.y * L.w));
    }
}

// Per (sample, segment, 64 neurons): (P_k, Q_k) from the segment's last
// event down to its first, each event's contributions, and the upstream
// gradient of the lane's spikes inside the segment.  The segment is staged
// as in the forward walks (sources in registers, decays and times in LDS);
// groups of kGrp events are walked from the last backwards with the next
// group's weights and records in flight, the dL/dW terms of a group added
// after its walk and its dL/dt terms summed over the lanes together
// (group_sum8).
constexpr int kRegPre = 4;

__global__ __launch_bounds__(kWave * kWalkWaves) void k_regg_walk(
    const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src, const int32_t* __restrict__ ev_n, int B,
    int E_max, int E_pad, const float* __restrict__ WT, int C_in, int N, int tiles, int S, int items, Model m,
    const Decay* __restrict__ dec, const float2* __restrict__ rec, const double2* __restrict__ coef,
    const double2* __restrict__ cin, const float* __restrict__ out_t, const int32_t* __restrict__ out_n,
    const int32_t* __restrict__ out_k, const double* __restrict__ scale, long long* __restrict__ gw,
    double* __restrict__ gtp, float* __restrict__ grad_spike)
{
    __shared__ double2 s_ad[kWalkWaves][kSeg];
    __shared__ float s_t[kWalkWaves][kSeg];
    WalkCoords c;
    if (!walk_coords<1>(items, tiles, S, ev_n, E_max, N, c)) return;
    const int n = c.n0, lane = c.lane, wv = (int)threadIdx.x / kWave;
    double2* lad = s_ad[wv];
    float* lt = s_t[wv];
    const Decay* d = dec + (size_t)c.b * E_pad;
    const float2* rb = rec + (size_t)c.b * (E_max + 1) * N + n;
    const float* tt = ev_t + (size_t)c.b * E_max;
    const Stage st = stage_segment(c, ev_src + (size_t)c.b * E_max + c.k0, d + c.k0, WT, C_in, N, lad, nullptr,
                                   nullptr);
#pragma unroll
    for (int h = 0; h < kSrcRegs; ++h) {
        const int e = h * kWave + lane;
        if (e < c.cnt) lt[e] = tt[c.k0 + e];
    }
    wave_lds_sync();
    const size_t bn = (size_t)c.b * N + n;
    const double2 G = c.live ? coef[bn] : make_double2(0.0, 0.0);
    const double sc = scale[0];
    const int k1 = c.k0 + c.cnt - 1;
    // (P, Q) at event k1: the later segments' part, and in the last segment
    // the open interval after the sample's last event
    const double2 ci = cin[((size_t)c.b * S + c.seg) * N + n];
    double Pm = ci.x, Ps = ci.y;
    const bool last = k1 + 1 == c.nb;
    const Decay en = last ? Decay{0.0, 0.0, 0.0, 0.0} : d[k1 + 1];
    RecTerm tn = rec_term(rb[(size_t)(k1 + 1) * N], G, en.A, en.D);     // the interval after event k1
    if (last) {
        Pm = fma(tn.mu, tn.em, Pm);
        Ps = fma(tn.mu, tn.es, Ps);
    }
    // the lane's spikes in this segment (out_k in [k0, k1]), last first; the
    // first kRegPre of them and their upstream gradients are held in
    // registers and written back after the walk, so that the walk itself
    // loads nothing but the next group's weights and records.  A wave where
    // some lane has more spikes in the segment (a burst) reads and updates
    // them in the walk instead.
    const float* ts = out_t + bn * (size_t)m.s_max;
    const int32_t* ks = out_k + bn * (size_t)m.s_max;
    float* gsp = grad_spike + bn * (size_t)m.s_max;
    int sp = 0;                                   // spikes with out_k <= k1 (out_k is non-decreasing)
    {
        int hi = c.live ? min(out_n[bn], m.s_max) : 0;
        while (sp < hi) {
            const int mid = (sp + hi) >> 1;
            if (ks[mid] <= k1) sp = mid + 1; else hi = mid;
        }
    }
    int pk[kRegPre];
    float pt[kRegPre], pg[kRegPre];
#pragma unroll
    for (int u = 0; u < kRegPre; ++u) {
        const int q = sp - 1 - u;
        const int kq = q >= 0 ? ks[q] : -1;
        const bool in = kq >= c.k0;
        pk[u] = in ? kq : -1;
        pt[u] = in ? ts[q] : 0.0f;
        pg[u] = in ? gsp[q] : 0.0f;
    }
    const int qx = sp - 1 - kRegPre;
    const bool burst = __ballot(qx >= 0 && ks[max(qx, 0)] >= c.k0) != 0ull;
    double* gt = gtp + ((size_t)c.tile * B + c.b) * E_max + c.k0;
    const double kap = m.kappa, sk = -(m.dth * m.inv_tm);
    auto load_rec = [&](int g, float2 (&r)[kGrp]) {
#pragma unroll
        for (int jj = 0; jj < kGrp; ++jj) r[jj] = rb[(size_t)(c.k0 + min(g * kGrp + jj, c.cnt - 1)) * N];
    };
    auto walk = [&](auto burst_tag) {
        constexpr bool kBurst = decltype(burst_tag)::value;
        int knext = kBurst && sp > 0 ? ks[sp - 1] : -1;
        // the walk of group g (its dL/dt terms ca and fixed-point dL/dW terms ga)
        auto group = [&](int g, const float (&w)[kGrp][1], const float2 (&r)[kGrp], double (&ca)[kGrp],
                         long long (&ga)[kGrp]) {
#pragma unroll
            for (int jj = kGrp - 1; jj >= 0; --jj) {
                const int e = g * kGrp + jj;
                ca[jj] = 0.0;
                ga[jj] = 0;
                if (e >= c.cnt) continue;
                const int k = c.k0 + e;
                const double2 ad = lad[e];
                const RecTerm t = rec_term(r[jj], G, ad.x, ad.y);        // the interval that event e closes
                double gk = (double)w[jj][0] * kap * (Pm * m.inv_tm - Ps * m.inv_ts);
                gk = fma(tn.mu, tn.vs, gk);              // adds 0 unless the argmax is that end
                gk = fma(t.mu, t.ve, gk);
                const long long gq = llrint(kap * (Pm - Ps) * sc);
                ca[jj] = c.live ? gk : 0.0;
                ga[jj] = c.live ? gq : 0ll;
                // spikes between events k - 1 and k: their upstream gradient
                // from P at event k
                if constexpr (kBurst) {
                    if (c.live && knext == k) {
                        const double tk = (double)lt[e];
                        while (sp > 0 && ks[sp - 1] == k) {
                            --sp;
                            gsp[sp] += (float)(sk * Pm * exp(-(tk - (double)ts[sp]) * m.inv_tm));
                        }
                        knext = sp > 0 ? ks[sp - 1] : -1;
                    }
                } else {
                    bool hit = false;
#pragma unroll
                    for (int u = 0; u < kRegPre; ++u) hit |= pk[u] == k;
                    if (__ballot(hit)) {
                        const double tk = (double)lt[e];
#pragma unroll
                        for (int u = 0; u < kRegPre; ++u)
                            if (pk[u] == k) pg[u] += (float)(sk * Pm * exp(-(tk - (double)pt[u]) * m.inv_tm));
                    }
                }
                if (e > 0) {
                    Pm = fma(t.mu, t.em, Pm * ad.x);
                    Ps = fma(t.mu, t.es, Ps * ad.y);
                }
                tn = t;
            }
        };
        // group g's dL/dW terms (zero terms included, so that every group
        // issues the same memory operations) and its dL/dt sums
        auto flush = [&](int g, const double (&ca)[kGrp], const long long (&ga)[kGrp]) {
            const int oreg = g * kGrp < kWave ? st.off[0] : st.off[kSrcRegs - 1];
#pragma unroll
            for (int jj = 0; jj < kGrp; ++jj) {
                const int roff = __builtin_amdgcn_readlane(oreg, (g * kGrp + jj) & (kWave - 1));
                atomicAdd((unsigned long long*)&gw[(size_t)(roff >> 2) + (size_t)n], (unsigned long long)ga[jj]);
            }
            const double sum = group_sum8(ca, lane);
            const int j = ((lane >> 5) & 1) * 4 + ((lane >> 4) & 1) * 2 + ((lane >> 3) & 1);
            if ((lane & 7) == 0 && g * kGrp + j < c.cnt) gt[g * kGrp + j] = sum;
        };
        // Groups from the last backwards with two groups' weights and records
        // in flight; a group's loads are issued before the atomics of the
        // group walked just before, so that no wait for loads waits for
        // atomics (the memory counter is in order).  Loads past the first
        // group re-read it.
        const int ng = (c.cnt + kGrp - 1) / kGrp;
        float wa[kGrp][1], wb[kGrp][1];
        float2 ra[kGrp], rbuf[kGrp];
        double ca[kGrp];
        long long ga[kGrp];
        load_grp<1>(st, (ng - 1) * kGrp, wa);
        load_rec(ng - 1, ra);
        load_grp<1>(st, max(ng - 2, 0) * kGrp, wb);
        load_rec(max(ng - 2, 0), rbuf);
        for (int g = ng - 1; g >= 0; g -= 2) {
            group(g, wa, ra, ca, ga);
            load_grp<1>(st, max(g - 2, 0) * kGrp, wa);
            load_rec(max(g - 2, 0), ra);
            flush(g, ca, ga);
            if (g < 1) break;
            group(g - 1, wb, rbuf, ca, ga);
            load_grp<1>(st, max(g - 3, 0) * kGrp, wb);
            load_rec(max(g - 3, 0), rbuf);
            flush(g - 1, ca, ga);
        }
    };
    if (burst) {
        walk(std::true_type{});
    } else {
        walk(std::false_type{});
#pragma unroll
        for (int u = 0; u < kRegPre; ++u)
            if (pk[u] >= 0) gsp[sp - 1 - u] = pg[u];
    }
}

// Fixed point -> float32 dL/dW; dL/dt summed over the tiles in order (0 past
// each sample's last event).
__global__ __launch_bounds__(256) void k_regg_convert(const long long* __restrict__ gw,
                                                     const double* __restrict__ scale, size_t nW,
                                                     float* __restrict__ grad_WT, const double* __restrict__ gtp,
                                                     const int32_t* __restrict__ ev_n, int B, int E_max, int tiles,
                                                     float* __restrict__ grad_ev_t)
{
    const size_t gtid = (size_t)blockIdx.x * blockDim.x + threadIdx.x, gs = (size_t)gridDim.x * blockDim.x;
    const double inv = 1.0 / scale[0];
    for (size_t x = gtid; x < nW; x += gs) grad_WT[x] = (float)((double)gw[x] * inv);
    if (!grad_ev_t) return;
    const size_t nT = (size_t)B * E_max;
    for (size_t x = gtid; x < nT; x += gs) {
        const int b = (int)(x / (size_t)E_max), k = (int)(x % (size_t)E_max);
        double g = 0.0;
        if (k < clamp_count(ev_n[b], E_max))
            for (int t = 0; t < tiles; ++t) g += gtp[(size_t)t * nT + x];
        grad_ev_t[x] = (float)g;
    }
}

struct RegGradLayout {
    RegLayout r;
    size_t rec, counts, gates, coef, musum, scale, local, cin, gw, gtp, total;
};

static RegGradLayout reg_grad_layout(int B, int E_max, int C_in, int N)
{
    RegGradLayout G;
    G.r = reg_layout(B, E_max, N);
    size_t off = G.r.total;
    auto take = [&](size_t bytes) { size_t o = off; off += (bytes + 255) & ~(size_t)255; return o; };
    const size_t BS = (size_t)B * G.r.f.S;
    const int tiles = (N + kWave - 1) / kWave;
    G.rec = take((size_t)B * ((size_t)E_max + 1) * N * sizeof(float2));
    G.counts = take((size_t)B * N * sizeof(double2));
    G.gates = take((size_t)N * sizeof(double2));
    G.coef = take((size_t)B * N * sizeof(double2));
    G.musum = take((size_t)B * N * sizeof(double));
    G.scale = take(sizeof(double));
    G.local = take(BS * N * sizeof(double4));
    G.cin = take(BS * N * sizeof(double2));
    G.gw = take((size_t)C_in * N * sizeof(long long));
    G.gtp = take((size_t)tiles * B * E_max * sizeof(double));
    G.total = off + 256;
    return G;
}

}  // namespace lif

extern "C" size_t lif_spike_count_reg_backward_workspace_size(int B, int E_max, int C_in, int N_out)
{
    if (B < 0 || E_max < 0 || C_in < 1 || N_out < 1) return 0;
    return lif::reg_grad_layout(B, E_max, C_in, N_out).total;
}

extern "C" int lif_spike_count_reg_backward(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B,
                                            int E_max, const float* WT, int C_in, int N_out, const lif_params* p,
                                            const float* out_t, const int32_t* out_n, const int32_t* out_k,
                                            double c_target, double lam_reg, double lam_over, float* loss,
                                            float* grad_spike, float* grad_WT, float* grad_ev_t, void* ws,
                                            size_t ws_bytes, lif_stream_t stream_)
{
    using namespace lif;
    int rc = validate_forward_args(ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, p, out_t, out_n, out_n);
    if (rc) return rc;
    if (!out_k || !grad_spike || !grad_WT || !ws || !(c_target > 0.0) || !isfinite(c_target) ||
        !isfinite(lam_reg) || !isfinite(lam_over))
        return LIF_ERR_ARG;
    const RegGradLayout G = reg_grad_layout(B, E_max, C_in, N_out);
    if (ws_bytes < G.total) return LIF_ERR_WORKSPACE;
    const int tl = (N_out + kWave - 1) / kWave;
    const size_t items_max = (size_t)B * G.r.f.S * tl;
    if (items_max > 0x7fffffff || B > 65535) return LIF_ERR_SIZE;
    hipStream_t stream = (hipStream_t)stream_;
    const Model m = make_model(*p);
    char* base = (char*)(((uintptr_t)ws + 255) & ~(uintptr_t)255);
    const RegLayout& R = G.r;
    FwdPtrs P{};
    P.dec = (Decay*)(base + R.f.dec);
    P.segm = (double2*)(base + R.f.segm);
    P.carry = (double2*)(base + R.f.carry);
    P.mask = (uint32_t*)(base + R.f.mask);
    P.counters = (uint32_t*)(base + R.f.counters);
    P.pool_count = P.counters;
    P.nwork = P.counters + (size_t)B * kCtr;
    P.listed = (uint32_t*)(base + R.f.listed);
    P.work = (uint32_t*)(base + R.f.work);
    P.pool = (double2*)(base + R.f.pool);
    double4* part = (double4*)(base + R.part);
    double* ub = (double*)(base + R.ub);
    double* ob = (double*)(base + R.ob);
    int32_t* st = (int32_t*)(base + R.status);
    float2* rec = (float2*)(base + G.rec);
    double2* counts = (double2*)(base + G.counts);
    double2* gates = (double2*)(base + G.gates);
    double2* coef = (double2*)(base + G.coef);
    double* musum = (double*)(base + G.musum);
    double* scale = (double*)(base + G.scale);
    double4* local = (double4*)(base + G.local);
    double2* cin = (double2*)(base + G.cin);
    long long* gw = (long long*)(base + G.gw);
    double* gtp = (double*)(base + G.gtp);
    const size_t nn = (size_t)B * N_out, nW = (size_t)C_in * N_out;
    const unsigned wblocks = (unsigned)((items_max + kWalkWaves - 1) / kWalkWaves);
    if (items_max > 0) {
        switch (pick_npl(WT, N_out)) {
        case 4: launch_walks<4>(R.f, P, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, m, st, false, nullptr, nullptr,
                                nullptr, nullptr, stream, false); break;
        case 2: launch_walks<2>(R.f, P, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, m, st, false, nullptr, nullptr,
                                nullptr, nullptr, stream, false); break;
        default: launch_walks<1>(R.f, P, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, m, st, false, nullptr,
                                 nullptr, nullptr, nullptr, stream, false); break;
        }
        TIMED_LAUNCH("reg_walk", k_reg_walk, dim3(wblocks), dim3(kWave * kWalkWaves), 0, stream, ev_t, ev_src, ev_n,
                     E_max, R.f.E_pad, WT, C_in, N_out, tl, R.f.S, (int)items_max, m, P.dec, P.carry, out_t, out_n,
                     out_k, part, rec, local);
    }
    if (nn)
        TIMED_LAUNCH("reg_reduce", k_reg_reduce, dim3((unsigned)((nn + 255) / 256)), dim3(256), 0, stream, part, ev_n,
                     B, E_max, N_out, R.f.S, m.th, ub, ob, nullptr, nullptr, counts);
    if (B > 0)
        TIMED_LAUNCH("reg_loss", k_reg_loss, dim3(1), dim3(kRegThreads), 0, stream, ub, ob, out_n, B, N_out, m.s_max,
                     c_target, loss, gates);
    size_t work = nW > nn ? nW : nn;
    size_t blocks = (work + 255) / 256;
    blocks = blocks < 1 ? 1 : (blocks > 2048 ? 2048 : blocks);
    TIMED_LAUNCH("regg_coef", k_regg_coef, dim3((unsigned)blocks), dim3(256), 0, stream, counts, gates, out_n, B,
                 N_out, m.s_max, c_target, lam_reg, lam_over, coef, musum, gw, nW);
    TIMED_LAUNCH("regg_scale", k_regg_scale, dim3(1), dim3(kRegThreads), 0, stream, musum, nn, ev_n, B, E_max,
                 m.kappa, scale);
    if (items_max > 0) {
        TIMED_LAUNCH("regg_carry", k_regg_carry, dim3((unsigned)tl, (unsigned)B), dim3(kWave), 0, stream, ev_n, E_max,
                     N_out, R.f.S, P.segm, local, coef, cin);
        TIMED_LAUNCH("regg_walk", k_regg_walk, dim3(wblocks), dim3(kWave * kWalkWaves), 0, stream, ev_t, ev_src, ev_n,
                     B, E_max, R.f.E_pad, WT, C_in, N_out, tl, R.f.S, (int)items_max, m, P.dec, rec, coef, cin, out_t,
                     out_n, out_k, scale, gw, gtp, grad_spike);
    }
    work = nW > (size_t)B * E_max ? nW : (size_t)B * E_max;
    blocks = (work + 255) / 256;
    blocks = blocks < 1 ? 1 : (blocks > 2048 ? 2048 : blocks);
    TIMED_LAUNCH("regg_convert", k_regg_convert, dim3((unsigned)blocks), dim3(256), 0, stream, gw, scale, nW, grad_WT,
                 gtp, ev_n, B, E_max, tl, grad_ev_t);
    return check_launch();
}

// ---------------------------------------------------------------------------
// Forward pass without a caller workspace: the workspace is a fixed array in
// device memory, one per GPU, held from the library's load until the process
// ends.  Its device address is looked up once per device (with that device
// current) and kept; host code passes only that address to kernels.
// ---------------------------------------------------------------------------
#include <mutex>

namespace lif {

constexpr size_t kScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices];

// The current device's address of the scratch array.
static int scratch_address(void** out)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return LIF_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return LIF_ERR_HIP;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return LIF_OK;
}

}  // namespace lif

extern "C" size_t lif_layer_forward_noalloc_max_bytes(void) { return lif::kScratchBytes; }

extern "C" int lif_layer_forward_noalloc(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B,
                                         int E_max, const float* WT, int C_in, int N_out, const lif_params* p,
                                         float* out_t, int32_t* out_n, float* out_i, int32_t* out_k,
                                         int32_t* status, lif_stream_t stream)
{
    using namespace lif;
    int rc = validate_forward_args(ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, p, out_t, out_n, status);
    if (rc) return rc;
    lif_params q = *p;
    // the layout without pool entries must fit; the default pool is cut to
    // what the array holds (sub-blocks past it take the rebuild path, with
    // identical results), a pool size the caller set must fit as it is
    if (fwd_layout(B, E_max, N_out, 0).total > kScratchBytes) return LIF_ERR_SIZE;
    if (q.pool_cap < 0) {
        size_t cap = fwd_layout(B, E_max, N_out, -1).pool_cap;
        if (cap > 0x7fffffff) cap = 0x7fffffff;
        size_t lo = 0, hi = cap;                      // largest fitting slice size
        while (lo < hi) {
            const size_t mid = hi - (hi - lo) / 2;
            if (fwd_layout(B, E_max, N_out, (int)mid).total <= kScratchBytes) lo = mid;
            else hi = mid - 1;
        }
        q.pool_cap = (int32_t)lo;
    }
    if (fwd_layout(B, E_max, N_out, q.pool_cap).total > kScratchBytes) return LIF_ERR_SIZE;
    void* ws = nullptr;
    rc = scratch_address(&ws);
    if (rc) return rc;
    return forward_impl(false, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, &q, out_t, out_n, out_i, out_k, status,
                        ws, kScratchBytes, (hipStream_t)stream);
}
