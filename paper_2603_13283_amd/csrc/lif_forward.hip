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
//                state entering every segment.
//   k_check      per (sample, segment, tile): re-walk from the carried state
//                with a no-crossing screen per inter-event interval
//                (screen_value).  Resets only lower V, so a sub-block of kSub
//                events whose no-reset trajectory passes every screen holds
//                no spike whatever happened before it; a flagged
//                sub-block stores its entering state and reserves a record.
//   k_records    per reserved record (lanes are the sub-block's intervals):
//                the no-reset states at every interval boundary of the
//                sub-block and each interval's crossing data; also resets the
//                outputs ahead of the resolve pass.
//   k_resolve    per (sample, neuron) with flagged sub-blocks: walks only
//                those, in time order.  Spikes found so far lower V by a
//                known decaying amount (the reset deficit), which corrects
//                the recorded states exactly.  Each interval is tested with
//                the interval rule (Sec. 3.2.2), the spike time is solved by
//                bracketed Newton (Appendix D.1), V is hard-reset and the
//                same interval is tested again from the spike (Appendix E.2).
// The sequential baseline k_sequential (Appendix E.3) runs the same interval
// rule and root solve one event at a time per (sample, neuron).
#include "lif_common.hpp"
#include "lif_host.hpp"
#include "lif_walk.hpp"

namespace lif {

// Record of one flagged sub-block of one neuron, in per-sample pools.  The
// check pass reserves it (one atomic per wave) and writes its header; the
// record pass k_records fills in, per interval j of the sub-block, the
// no-reset state (V, I) at the interval start and the interval's crossing
// data.  With the reset deficit of the spikes found so far these give the
// true state at every interval boundary in O(1), so the resolve pass can test
// all intervals of the sub-block at once.
struct alignas(16) Record {
    double2 s[kSub + 1];    // s[j]: state at the start of interval j (after event j - 1); in the
                            // sub-block holding the sample's last event, s[cnt]: the state after it
    double crit[kSub + 1];  // interval j crosses iff the deficit at its start is <= crit[j] (< 0: never);
                            // entry kSub: the open interval after the sample's last event (in the
                            // record of the sub-block that holds it)
    double hi[kSub + 1];    // right end of interval j's root bracket (u* or its length)
    double fhi[kSub + 1];   // h(hi) of interval j (F(hi) = fhi - deficit)
    int32_t kq0, cnt, n;    // first event of the sub-block (index in the sample), events in it, neuron
    int32_t pad_[3];
};
static_assert(sizeof(Record) % 16 == 0, "record layout");
constexpr uint32_t kNoSlot = 0xffffffffu;

// Per-sample counters (record-pool use, work-list length) each take their
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
    uint32_t* __restrict__ counters, size_t n_counters, uint32_t* __restrict__ listed, size_t nn)
{
    {
        // resets for the later passes: status words, per-sample counters,
        // listed flags (grid-stride over every thread)
        const size_t gt = (size_t)blockIdx.x * blockDim.x + threadIdx.x, gs = (size_t)gridDim.x * blockDim.x;
        if (gt < LIF_STATUS_WORDS) status[gt] = 0;
        for (size_t i = gt; i < n_counters; i += gs) counters[i] = 0u;
        for (size_t i = gt; i < nn; i += gs) listed[i] = 0u;
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
// again from its incoming state, writing the carries.
constexpr int kCarryWaves = 8;
constexpr int kCarryBatch = 16;

__global__ __launch_bounds__(kWave * kCarryWaves) void k_carry(
    const int32_t* __restrict__ ev_n, int B, int E_max, int N, int tiles, int S, const double2* __restrict__ segm,
    const double2* __restrict__ agg, double2* __restrict__ carry)
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
// (up to t_end).  A flagged (sub-block, neuron) stores its entering state
// (U, J) in ent and sets a bit in the neuron's sub-block mask of the segment.
// At the end of the item the wave reserves records for all its flagged
// sub-blocks with one atomic on the sample's pool counter, in lane order, so
// that the records of one (segment, neuron) are consecutive: the mask word
// of the pair holds the sub-block bits and the pool offset of its first
// record, and the record of a flagged sub-block is that offset plus the
// number of flagged sub-blocks before it (none past the pool capacity: the
// resolve pass then rebuilds that sub-block's states from ent itself).  The
// wave writes the records' headers; the first segment to flag a neuron
// appends it to the sample's work list.
__global__ __launch_bounds__(kWave * kWalkWaves) void k_check(
    const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src, const int32_t* __restrict__ ev_n, int E_max,
    int E_pad, const float* __restrict__ WT, int C_in, int N, int tiles, int S, int items, Model m,
    const Decay* __restrict__ dec, const double2* __restrict__ carry, double2* __restrict__ ent,
    uint2* __restrict__ mask, Record* __restrict__ pool,
    uint32_t* __restrict__ pool_count, uint32_t pool_cap, uint32_t* __restrict__ listed,
    uint32_t* __restrict__ work, uint32_t* __restrict__ nwork)
// work: per-sample lists of the neurons with flagged sub-blocks (capacity N
// each); nwork: per-sample list lengths.
{
    constexpr int NPL = 1;                  // one neuron per lane (occupancy)
    __shared__ double2 s_ad[kWalkWaves][kSeg];
    __shared__ double s_lk[kWalkWaves][kSeg];
    __shared__ double s_gk[kWalkWaves][kGrpPerSeg];
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
        const size_t srow = (((size_t)c.b * S + c.seg) * kSubPerSeg + q) * N + c.n0;
#pragma unroll
        for (int i = 0; i < NPL; ++i)
            if (c.live && z[i] >= m.thk_lo) {
                ent[srow + i] = make_double2(U0[i], J0[i]);
                msk[i] |= 1u << q;
            }
    }
    // Records of the wave's flagged sub-blocks: one reservation, slots in
    // lane order (exclusive prefix sum of the per-lane counts).
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
            if (c.live) mask[row + i] = make_uint2(msk[i], base);
            for (uint32_t mm = msk[i]; mm; mm &= mm - 1u) {
                if (base < pool_cap) {
                    Record* r = pool + ((size_t)c.b * pool_cap + base);
                    const int kq0 = c.k0 + __builtin_ctz(mm) * kSub;
                    r->kq0 = kq0;
                    r->cnt = min(kSub, c.nb - kq0);
                    r->n = c.n0 + i;
                }
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
// ---------------------------------------------------------------------------
// Resolve pass: one workgroup of two waves per neuron that has flagged
// sub-blocks (a work list built by the check pass).  Intervals outside
// flagged sub-blocks provably hold no spike.  The flagged sub-blocks are
// taken in time order:
//   * Candidate list: per chunk of kChunkEv events, the sub-block masks (one
//     to two segments per lane) are compacted into
//     a time-ordered list in LDS with one wave prefix sum, with the record
//     slot of every candidate.
//   * Windows of kWinCand candidates in two LDS buffers: the staging wave
//     (wave 1) loads and commits window w + 1 into one buffer while the chain
//     wave (wave 0) resolves window w from the other, so the loads and LDS
//     writes of a window stay off the serial chain.  One barrier per window.
//   * Steps of kWave / kSub = 4 candidates: lane l takes interval l % kSub of
//     candidate l / kSub, so time order is lane order.  Each interval
//     carries its crossing data (k_records): it crosses iff the reset
//     deficit at its start is <= crit.  A round takes the earliest crossing
//     interval (ballot), solves its spike time (root_h) on its lane, emits
//     the spike and raises that interval's own deficit (so it is tested again
//     for a second spike, Appendix E.2 restart); every later interval takes
//     the new deficit with one exponential.  Rounds repeat until no interval
//     of the step crosses.
//   * The open interval after the sample's last event is one more step (one
//     lane) after the last window.
//   * Spikes are buffered in LDS and written out kWave at a time.
// The resolve kernel runs few waves per compute unit, so nearly all of its
// code is fetched cold: every path is written once (no unrolled copies of
// the solver or of the rare rebuild of sub-blocks without a record).
// Wave-uniform state: spike count, reset deficit dref right after the
// latest spike, at time tref.
// ---------------------------------------------------------------------------
constexpr int kChunkEv = 8192;                   // events per chunk of the candidate list
constexpr int kChunkSeg = kChunkEv / kSeg;       // segments per chunk
constexpr int kSegPerLane = kChunkSeg / kWave;   // mask words per lane
static_assert(kChunkSeg % kWave == 0 && kSubPerSeg <= 8, "chunk layout; 3-bit sub-block field of a candidate");
constexpr int kCandCap = kChunkSeg * kSubPerSeg; // candidates of one chunk
constexpr int kStep = kWave / kSub;              // candidates per step
constexpr int kWinCand = 16;                     // candidates per window
constexpr int kWinIv = kWinCand * kSub;          // intervals per window
constexpr int kIvPerLane = kWinIv / kWave;       // window intervals staged by each lane
constexpr int kWinSteps = kWinCand / kStep;
constexpr int kOpenIv = kWinIv;                  // window slot of the open interval

// One window, interval i = candidate * kSub + j; slot kOpenIv: the open
// interval.
struct WinBuf {
    double crit[kWinIv + 1], hi[kWinIv + 1], fhi[kWinIv + 1];
    double2 s0[kWinIv + 1];                      // (V0, I0)
    double t0[kWinIv + 1];                       // interval start
    int32_t kev[kWinIv + 1];                     // index of the event that closes the interval (ev_n[b]: open)
};

struct ResolveLds {
    uint32_t cand[kCandCap];                     // (segment in chunk << 3) | sub-block
    uint32_t slot[kCandCap];                     // record slot of each candidate (kNoSlot: none)
    WinBuf win[2];
    double sp_t0[kWave], sp_y[kWave];            // spike buffer: interval start, e^{-u/tm},
    float si[kWave];                             // I at the spike,
    int32_t sk[kWave];                           // events consumed before the spike
    int ntot;                                    // candidates of the chunk (chain wave -> both)
    int stop[2];                                 // capped after window w (slot w % 2)
};
constexpr int kResolveWaves = 2;

// Crossing data of one interval of length L that starts in the no-reset
// state (V0, I0) and ends with V1 (A, D: its decays): the interval reaches
// the threshold iff the reset deficit at its start is <= crit (crit < 0:
// never), by interval_max's test D a <= g; the spike then lies in
// (lo, hi] with F(hi) = fhi - deficit.  Zero-length intervals never cross.
// k_records and the resolve pass (sub-blocks without a record)
// both evaluate it; with floating-point contraction off here and in
// interval_max, every inlined copy performs the same IEEE operations, so
// both give the same bits whichever path a sub-block takes.
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

// States of interval j of a sub-block (events kq0 .. kq0 + cnt - 1 of the
// sample) from the sub-block's entering no-reset state (U, J): the lane walks
// events 0 .. j, taking the state at the interval start (after event j - 1)
// and, after event j, V at the interval end and J.  The record pass and the
// resolve pass's rebuild of sub-blocks without a record both call it, so the
// two give the same bits.
struct IvStates {
    double V0, I0, V1, J1;
};

template <bool kHoist>
__device__ __forceinline__ IvStates subblock_walk(const Model& m, double U, double J, int kq0, int cnt, int j, int n,
                                                  int N, int C_in, const int32_t* __restrict__ src,
                                                  const Decay* __restrict__ d, const float* __restrict__ WT)
{
    IvStates r{0.0, 0.0, 0.0, 0.0};
    const int last = max(cnt - 1, 0);
    if constexpr (kHoist) {
        // every load first (independent, clamped to the sub-block), then the walk
        int sc[kSub];
#pragma unroll
        for (int e = 0; e < kSub; ++e) sc[e] = clamp_src(src[kq0 + min(e, last)], C_in);
        float wv[kSub];
        double2 ad[kSub];
#pragma unroll
        for (int e = 0; e < kSub; ++e) {
            wv[e] = WT[(size_t)sc[e] * (size_t)N + n];
            const Decay dk = d[kq0 + min(e, last)];
            ad[e] = make_double2(dk.A, dk.D);
        }
#pragma unroll
        for (int e = 0; e < kSub; ++e) {
            if (e == j) {
                r.V0 = v_of(m, U, J);
                r.I0 = J;
            }
            if (e <= j && e < cnt) {
                const double w = (double)wv[e];
                U = fma(ad[e].x, U, w);
                J = fma(ad[e].y, J, w);
            }
        }
    } else {
        // the same operations, one event at a time (few registers)
        for (int e = 0; e < kSub; ++e) {
            if (e == j) {
                r.V0 = v_of(m, U, J);
                r.I0 = J;
            }
            const int k = kq0 + min(e, last);
            const bool step_in = e <= j && e < cnt;
            const double w = step_in ? (double)WT[(size_t)clamp_src(src[k], C_in) * (size_t)N + n] : 0.0;
            const Decay dk = d[k];
            if (step_in) {
                U = fma(dk.A, U, w);
                J = fma(dk.D, J, w);
            }
        }
    }
    r.V1 = v_of(m, U, J);
    r.J1 = J;
    return r;
}

// k_records: the states and crossing data of every reserved record, in
// parallel (lanes are intervals, 4 records per wave), and of the open
// interval in the record of each sample's last sub-block.  This keeps the
// sub-block walks and the closed-form maximum of each interval (a log and an
// exp) off the resolve pass's per-neuron serial chain.  Grid: (blocks per
// sample, B); the records of sample blockIdx.y are spread over that sample's
// blocks.
__global__ __launch_bounds__(256) void k_records(const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src,
                                                 const int32_t* __restrict__ ev_n, int E_max, int E_pad, int S,
                                                 const float* __restrict__ WT, int C_in, int N, Model m,
                                                 const Decay* __restrict__ dec, const double2* __restrict__ ent,
                                                 Record* __restrict__ pool, const uint32_t* __restrict__ pool_count,
                                                 uint32_t pool_cap, int32_t* __restrict__ out_n, size_t nn,
                                                 float* __restrict__ out_t, float* __restrict__ out_i,
                                                 int32_t* __restrict__ out_k, size_t n_out, int B,
                                                 int32_t* __restrict__ status)
{
    if (blockIdx.x == gridDim.x - 1 && blockIdx.y == gridDim.y - 1 && threadIdx.x >= blockDim.x - kWave) {
        // status words fixed once the check pass has run (the only writer of
        // these words in the call): events consumed, flagged sub-blocks,
        // sub-blocks past the pool's capacity
        const int l = (int)threadIdx.x % kWave;
        unsigned long long ev = 0, fl = 0, fb = 0;
        for (int bb = l; bb < B; bb += kWave) {
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
        if (l == 0) {
            auto sat = [](unsigned long long x) { return (int32_t)(x > 0x7fffffffull ? 0x7fffffffull : x); };
            status[LIF_ST_EVENTS] = sat(ev);
            status[LIF_ST_CAND_BLOCKS] = sat(fl);
            status[LIF_ST_WALKED_BLOCKS] = sat(fl);
            status[LIF_ST_POOL_FALLBACK] = sat(fb);
        }
    }
    {
        // outputs reset ahead of the resolve pass (it writes only the
        // neurons that fire): counts 0, times +inf, currents and event
        // counts 0
        const size_t gs = (size_t)gridDim.x * gridDim.y * blockDim.x;
        const size_t gt = ((size_t)blockIdx.y * gridDim.x + blockIdx.x) * blockDim.x + threadIdx.x;
        for (size_t i = gt; i < nn; i += gs) out_n[i] = 0;
        for (size_t i = gt; i < n_out; i += gs) {
            out_t[i] = INFINITY;
            if (out_i) out_i[i] = 0.0f;
            if (out_k) out_k[i] = 0;
        }
    }
    const int lane = (int)threadIdx.x % kWave;
    const int j = lane % kSub;
    const uint32_t gw = (blockIdx.x * blockDim.x + threadIdx.x) / kWave;
    const uint32_t nw = gridDim.x * blockDim.x / kWave;
    constexpr uint32_t kRecPerWave = kWave / kSub;
    const int b = blockIdx.y;
    const int nb = clamp_count(ev_n[b], E_max);
    const uint32_t used = min(pool_count[(size_t)b * kCtr], pool_cap);
    const float* tt = ev_t + (size_t)b * E_max;
    const int32_t* src = ev_src + (size_t)b * E_max;
    const Decay* d = dec + (size_t)b * E_pad;
    for (uint32_t r0 = gw * kRecPerWave; r0 < used; r0 += nw * kRecPerWave) {
        const uint32_t r = r0 + (uint32_t)(lane / kSub);
        if (r >= used) continue;
        Record* rec = pool + (size_t)b * pool_cap + r;
        const int kq0 = rec->kq0, cnt = rec->cnt, n = rec->n;
        if (j >= cnt || kq0 < 0 || kq0 + j >= nb || n < 0 || n >= N) continue;
        const int seg = kq0 / kSeg, q = (kq0 % kSeg) / kSub;
        const double2 e0 = ent[(((size_t)b * S + seg) * kSubPerSeg + q) * N + n];
        const IvStates v = subblock_walk<true>(m, e0.x, e0.y, kq0, cnt, j, n, N, C_in, src, d, WT);
        const int k = kq0 + j;
        const double t0 = k > 0 ? (double)tt[k - 1] : 0.0;
        double crit, hi, fhi;
        crossing_data(m, v.V0, v.I0, v.V1, (double)tt[k] - t0, d[k].A, d[k].D, crit, hi, fhi);
        rec->s[j] = make_double2(v.V0, v.I0);
        rec->crit[j] = crit;
        rec->hi[j] = hi;
        rec->fhi[j] = fhi;
        if (k == nb - 1) {
            // the open interval after the sample's last event
            open_interval_data(m, v.V1, v.J1, m.t_end - (double)tt[k], crit, hi, fhi);
            rec->s[j + 1] = make_double2(v.V1, v.J1);
            rec->crit[kSub] = crit;
            rec->hi[kSub] = hi;
            rec->fhi[kSub] = fhi;
        }
    }
}

__device__ __forceinline__ int rl_int(int v, int l) { return __builtin_amdgcn_readlane(v, l); }

__device__ __forceinline__ double rl_double(double v, int l)
{
    unsigned long long u = (unsigned long long)__double_as_longlong(v);
    unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)u, l);
    unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(u >> 32), l);
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// Loads of window interval h kWave + lane: candidate c = c0 + h kStep +
// lane / kSub, interval j = lane % kSub (unconditional loads from clamped
// addresses; nothing derived from the loaded values here).
struct StageIv {
    double crit, hi, fhi;
    double2 s0;
    float tp;
};

__device__ __forceinline__ StageIv stage_load(const ResolveLds& sh, int c, int tot, int seg0, int nb, int j,
                                              const float* __restrict__ tt, const Record* __restrict__ pool)
{
    StageIv v;
    const int cc = min(c, tot - 1);
    const uint32_t cw = sh.cand[cc];
    const uint32_t slot = sh.slot[cc];
    const int kq0 = (seg0 + (int)(cw >> 3)) * kSeg + (int)(cw & 7u) * kSub;
    const int k = min(kq0 + j, nb - 1);
    v.tp = tt[max(k - 1, 0)];
    const Record* rec = pool + (slot != kNoSlot ? slot : 0u);   // pool holds at least one record
    v.s0 = rec->s[j];
    v.crit = rec->crit[j];
    v.hi = rec->hi[j];
    v.fhi = rec->fhi[j];
    return v;
}

// Sub-blocks without a record (the pool was full): rebuild the window's
// intervals from the sub-blocks' entering states (U, J) with subblock_walk,
// as the record pass does, then the crossing data (and the open interval's,
// on the lane of the sample's last event).
__device__ __forceinline__ void rebuild_window(const ResolveLds& sh, WinBuf& w, const Model& m, int c0, int tot,
                                               int seg0, int b, int n, int nb, int S, int N, int C_in,
                                               const float* __restrict__ tt, const int32_t* __restrict__ src,
                                               const Decay* __restrict__ d, const float* __restrict__ WT,
                                               const double2* __restrict__ ent)
{
    const int lane = (int)threadIdx.x % kWave;
    const int j = lane % kSub;
    for (int h = 0; h < kIvPerLane; ++h) {
        const int c = c0 + h * kStep + lane / kSub;
        const bool in = c < tot;
        const int cc = min(c, tot - 1);
        const bool fb = in && sh.slot[cc] == kNoSlot;
        if (!__ballot(fb)) continue;
        const uint32_t cw = sh.cand[cc];
        const int seg = seg0 + (int)(cw >> 3), q = (int)(cw & 7u);
        const int kq0 = seg * kSeg + q * kSub, cnt = min(kSub, nb - kq0);
        const double2 e0 = fb ? ent[(((size_t)b * S + seg) * kSubPerSeg + q) * N + n] : make_double2(0.0, 0.0);
        const IvStates v = subblock_walk<true>(m, e0.x, e0.y, kq0, cnt, j, n, N, C_in, src, d, WT);
        if (fb && j < cnt) {
            const int i = h * kWave + lane;
            const int k = kq0 + j;
            const double t0 = k > 0 ? (double)tt[k - 1] : 0.0;
            const Decay dk = d[k];
            crossing_data(m, v.V0, v.I0, v.V1, (double)tt[k] - t0, dk.A, dk.D, w.crit[i], w.hi[i], w.fhi[i]);
            w.s0[i] = make_double2(v.V0, v.I0);
            if (k == nb - 1) {
                open_interval_data(m, v.V1, v.J1, m.t_end - (double)tt[k], w.crit[kOpenIv], w.hi[kOpenIv],
                                   w.fhi[kOpenIv]);
                w.s0[kOpenIv] = make_double2(v.V1, v.J1);
            }
        }
    }
}


// Wave-uniform resolve state of one neuron: the reset deficit of the spikes
// so far is D(t) = dref e^{-(t - tref)/tm} for t after the latest spike,
// with tref the start of the interval that spike lies in (the deficit is
// carried in that interval's frame, so no spike time is needed on the chain).
struct Chain {
    int ns;              // spikes so far
    double dref, tref;
    bool capped;
};

// Spikes [from, to) from the LDS buffer to the outputs (coalesced); the
// spike times t0 - tm ln y are taken here, 64 at a time, off the per-spike
// chain.
__device__ __forceinline__ void flush_spikes(ResolveLds& sh, const Model& m, int from, int to, float* __restrict__ st,
                                             float* __restrict__ si, int32_t* __restrict__ sk)
{
    const int lane = (int)threadIdx.x;
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

// Rounds over one step (see the section comment): lane l takes window
// interval i0 + l if l < nlanes.  Each lane holds the deficit Dl at its
// interval's start; an interval crosses iff Dl <= crit.  The spike-time
// solve of a round runs wave-uniform on the crossing interval's data
// (broadcast from its lane), so its iterations branch on scalars.
__device__ __forceinline__ void resolve_step(ResolveLds& sh, const WinBuf& w, const Model& m, int i0, int nlanes,
                                             Chain& ch, float* __restrict__ st, float* __restrict__ si,
                                             int32_t* __restrict__ sk)
{
    const int lane = (int)threadIdx.x;
    const int i = lane < nlanes ? i0 + lane : i0;
    const double crit = w.crit[i];
    const double t0 = w.t0[i];
    double Dl = ch.ns > 0 ? ch.dref * exp(-(t0 - ch.tref) * m.inv_tm) : 0.0;
    bool pend = lane < nlanes && crit >= 0.0 && Dl <= crit;
    unsigned long long cm = __ballot(pend);
    if (!cm) return;
    const double2 s0 = w.s0[i];
    const double hi = w.hi[i], fhi = w.fhi[i];
    double ylo = 1.0;
    for (;;) {
        const int kl = __ffsll((long long)cm) - 1;
        const double V0k = rl_double(s0.x, kl), I0k = rl_double(s0.y, kl), Dk = rl_double(Dl, kl);
        const double t0k = rl_double(t0, kl), hik = rl_double(hi, kl), fhik = rl_double(fhi, kl);
        const double ylok = rl_double(ylo, kl);
        const double kI = m.kappa * I0k;
        // after a spike inside the interval the raised deficit keeps F < 0
        // on all of [0, u], so the general solver may bracket from the
        // interval start; the polynomial solver starts from the spike (ylo)
        const SpikeY sp = solve_spike_y(m, V0k - Dk + kI, kI, 0.0, ylok, V0k - m.th - Dk, hik, fhik - Dk);
        if (lane == 0) {
            sh.sp_t0[ch.ns % kWave] = t0k;
            sh.sp_y[ch.ns % kWave] = sp.y;
            sh.si[ch.ns % kWave] = (float)(I0k * (sp.E2 * sp.y));
            sh.sk[ch.ns % kWave] = w.kev[i0 + kl];
        }
        // the deficit in interval kl's frame
        const double Dnew = Dk + m.dth * sp.E1;
        ++ch.ns;
        ch.dref = Dnew;
        ch.tref = t0k;
        if (ch.ns % kWave == 0) flush_spikes(sh, m, ch.ns - kWave, ch.ns, st, si, sk);
        if (ch.ns >= m.s_max) { ch.capped = true; return; }
        // interval kl is tested again with the raised deficit (a second spike
        // in it); later intervals take the new deficit; earlier ones are done
        const double Dlater = Dnew * exp(-(t0 - t0k) * m.inv_tm);
        Dl = lane == kl ? Dnew : Dlater;
        ylo = lane == kl ? sp.y : ylo;
        pend = pend && lane >= kl && Dl <= crit;
        cm = __ballot(pend);
        if (!cm) return;
    }
}

// The staging wave's part of window c0 / kWinCand: its intervals' loads,
// committed to buffer w, then the rebuild of its sub-blocks without a record.
__device__ __forceinline__ void stage_window(const ResolveLds& sh, WinBuf& w, const Model& m, int c0, int tot,
                                             int seg0, int b, int n, int nb, int S, int N, int C_in,
                                             const float* __restrict__ tt, const int32_t* __restrict__ src,
                                             const Decay* __restrict__ d, const float* __restrict__ WT,
                                             const double2* __restrict__ ent, const Record* __restrict__ pool)
{
    const int lane = (int)threadIdx.x % kWave;
    const int j = lane % kSub, r = lane / kSub;
    StageIv nx[kIvPerLane];
#pragma unroll
    for (int h = 0; h < kIvPerLane; ++h) nx[h] = stage_load(sh, c0 + h * kStep + r, tot, seg0, nb, j, tt, pool);
#pragma unroll
    for (int h = 0; h < kIvPerLane; ++h) {
        const int c = c0 + h * kStep + r;
        const int i = h * kWave + lane;
        const uint32_t cw = sh.cand[min(c, tot - 1)];
        const int kq0 = (seg0 + (int)(cw >> 3)) * kSeg + (int)(cw & 7u) * kSub;
        const bool valid = c < tot && kq0 + j < nb;
        w.crit[i] = valid ? nx[h].crit : -1.0;
        w.hi[i] = nx[h].hi;
        w.fhi[i] = nx[h].fhi;
        w.s0[i] = nx[h].s0;
        w.t0[i] = kq0 + j > 0 ? (double)nx[h].tp : 0.0;
        w.kev[i] = kq0 + j;
    }
    static_assert(kWinCand <= kWave, "one lane per candidate of the window");
    if (__ballot(sh.slot[min(c0 + lane % kWinCand, tot - 1)] == kNoSlot))
        rebuild_window(sh, w, m, c0, tot, seg0, b, n, nb, S, N, C_in, tt, src, d, WT, ent);
}

// Both waves of the workgroup call this for the same neuron and pass the
// same barriers (every loop bound is workgroup-uniform: candidate counts and
// the capped flag are exchanged through LDS).  Returns the spike count on the
// chain wave, 0 on the staging wave.
__device__ int resolve_neuron(ResolveLds& sh, int b, int n, const float* __restrict__ ev_t,
                              const int32_t* __restrict__ ev_src, const int32_t* __restrict__ ev_n, int E_max,
                              const float* __restrict__ WT, int C_in, int N, int E_pad, int S, const Model& m,
                              const Decay* __restrict__ dec, const double2* __restrict__ ent,
                              const uint2* __restrict__ mask, uint32_t pool_cap,
                              const Record* __restrict__ pool, float* __restrict__ out_t, int32_t* __restrict__ out_n,
                              float* __restrict__ out_i, int32_t* __restrict__ out_k)
{
    const int lane = (int)threadIdx.x % kWave;
    const bool chain = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave)) == 0;   // wave-uniform
    // the first chunk's mask words are loaded together with the event count
    // (words past the sample's segments are dropped below)
    uint2 mw[kSegPerLane];
#pragma unroll
    for (int h = 0; h < kSegPerLane; ++h) {
        const int sj = lane * kSegPerLane + h;
        mw[h] = chain && sj < S ? mask[((size_t)b * S + sj) * N + n] : make_uint2(0u, 0u);
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

    Chain ch{0, 0.0, 0.0, false};
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
                if (seg0 > 0) mw[h] = sj < Sb ? mask[((size_t)b * S + sj) * N + n] : make_uint2(0u, 0u);
                mv[h] = sj < Sb ? mw[h].x : 0u;
                pc += __popc(mv[h]);
            }
            int ex = pc;
#pragma unroll
            for (int off = 1; off < kWave; off <<= 1) {
                int v = __shfl_up(ex, off, kWave);
                if (lane >= off) ex += v;
            }
            const int ctot = rl_int(ex, kWave - 1);
            ex -= pc;
            // candidates and their record slots (consecutive per segment)
            int o = ex;
#pragma unroll
            for (int h = 0; h < kSegPerLane; ++h) {
                uint32_t mm = mv[h], rel = mw[h].y;
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
        if (tot > 0) {
            // the open interval is taken after the window holding the sample's
            // last sub-block, when that sub-block is flagged (it is the last
            // candidate of the last chunk)
            const uint32_t cwl = (uint32_t)__builtin_amdgcn_readfirstlane((int)sh.cand[tot - 1]);
            const bool open_here = has_open && (seg0 + (int)(cwl >> 3)) * kSeg + (int)(cwl & 7u) * kSub + kSub >= nb;
            const int nwin = (tot + kWinCand - 1) / kWinCand;
            if (!chain) {
                if (open_here) {
                    // the open interval's data, from the last candidate's
                    // record, in slot kOpenIv of both buffers (the windows do
                    // not overwrite it; a rebuild of the last sub-block does)
                    const uint32_t slot = (uint32_t)__builtin_amdgcn_readfirstlane((int)sh.slot[tot - 1]);
                    const int kq0 = (seg0 + (int)(cwl >> 3)) * kSeg + (int)(cwl & 7u) * kSub;
                    const Record* rec = pool + (slot != kNoSlot ? slot : 0u);
                    const double oc = rec->crit[kSub], oh = rec->hi[kSub], of = rec->fhi[kSub];
                    const double2 os = rec->s[min(nb - kq0, kSub)];
                    const double ot = (double)tt[nb - 1];
                    if (lane < 2) {
                        WinBuf& w = sh.win[lane];
                        w.crit[kOpenIv] = slot != kNoSlot ? oc : -1.0;
                        w.hi[kOpenIv] = oh;
                        w.fhi[kOpenIv] = of;
                        w.s0[kOpenIv] = os;
                        w.t0[kOpenIv] = ot;
                        w.kev[kOpenIv] = nb;
                    }
                }
                stage_window(sh, sh.win[0], m, 0, tot, seg0, b, n, nb, S, N, C_in, tt, src, d, WT, ent, pool);
            }
            __syncthreads();
            for (int wi = 0; wi < nwin; ++wi) {
                if (!chain) {
                    if (wi + 1 < nwin)
                        stage_window(sh, sh.win[(wi + 1) & 1], m, (wi + 1) * kWinCand, tot, seg0, b, n, nb, S, N,
                                     C_in, tt, src, d, WT, ent, pool);
                } else {
                    // the window's steps, then (last window) the open interval as one more
                    const WinBuf& w = sh.win[wi & 1];
                    const int c0 = wi * kWinCand;
                    const int steps = min(kWinSteps, (tot - c0 + kStep - 1) / kStep);
                    const int nsteps = steps + (wi == nwin - 1 && open_here ? 1 : 0);
                    for (int g = 0; g < nsteps && !ch.capped; ++g)
                        resolve_step(sh, w, m, g < steps ? g * kWave : kOpenIv, g < steps ? kWave : 1, ch, st, si, sk);
                    if (lane == 0) sh.stop[wi & 1] = ch.capped ? 1 : 0;
                }
                __syncthreads();              // window wi + 1 staged, window wi free
                stop = __builtin_amdgcn_readfirstlane(sh.stop[wi & 1]) != 0;
                if (stop) break;
            }
        }
        __syncthreads();                      // the list is rewritten by the next chunk
    }
    if (!chain) return 0;
    flush_spikes(sh, m, ch.ns - ch.ns % kWave, ch.ns, st, si, sk);
    if (lane == 0) out_n[idx] = ch.ns;
    return ch.ns;
}

// Work-list driven: the per-sample lists of neurons built by k_check are
// taken as one concatenated list, entry w by workgroup w mod gridDim.x, so
// that samples with many listed neurons spread over the whole grid.  Status
// counts are added once per workgroup.
__global__ __launch_bounds__(kWave * kResolveWaves) void k_resolve(const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src,
                                                   const int32_t* __restrict__ ev_n, int B, int E_max,
                                                   const float* __restrict__ WT, int C_in, int N, int E_pad, int S,
                                                   Model m, const Decay* __restrict__ dec,
                                                   const double2* __restrict__ ent,
                                                   const uint2* __restrict__ mask, uint32_t pool_cap,
                                                   const Record* __restrict__ pool,
                                                   const uint32_t* __restrict__ work, const uint32_t* __restrict__ nwork,
                                                   float* __restrict__ out_t, int32_t* __restrict__ out_n,
                                                   float* __restrict__ out_i, int32_t* __restrict__ out_k,
                                                   int32_t* __restrict__ status)
{
    __shared__ ResolveLds sh;
    // spikes and capped neurons of this workgroup's neurons, added to the
    // status words once at its end (no-return atomics: the wave does not
    // wait for them)
    unsigned long long spikes = 0;
    uint32_t capped = 0;
    const int lane = (int)threadIdx.x % kWave;
    // Both waves walk the list the same way.  Running sum of the list lengths over groups of 64 samples (one load
    // per lane, a wave prefix sum): entry w of the concatenated lists belongs
    // to the first sample whose running sum exceeds w.
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
        // wave-uniform by construction; readfirstlane lets the compiler
        // treat everything derived from it as uniform (scalar branches)
        const uint32_t bn = (uint32_t)__builtin_amdgcn_readfirstlane((int)work[(size_t)b * N + (w - before)]);
        const int ns = resolve_neuron(sh, (int)(bn / (uint32_t)N), (int)(bn % (uint32_t)N), ev_t, ev_src, ev_n,
                                      E_max, WT, C_in, N, E_pad, S, m, dec, ent, mask, pool_cap, pool, out_t, out_n,
                                      out_i, out_k);
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
// parallel path fills the same words inside its record and resolve passes.
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
__global__ __launch_bounds__(64) void k_sequential(const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src,
                                                   const int32_t* __restrict__ ev_n, int B, int E_max,
                                                   const float* __restrict__ WT, int C_in, int N, Model m,
                                                   int E_pad, const Decay* __restrict__ dec, float* __restrict__ out_t,
                                                   int32_t* __restrict__ out_n, float* __restrict__ out_i,
                                                   int32_t* __restrict__ out_k)
{
    const size_t idx_raw = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const bool live = idx_raw < (size_t)B * (size_t)N;
    const size_t idx = live ? idx_raw : 0;            // lanes past the end run neuron 0 and write nothing
    int b = (int)(idx / (size_t)N), n = (int)(idx % (size_t)N);
    int nb = clamp_count(ev_n[b], E_max);
    const float* tt = ev_t + (size_t)b * E_max;
    const int32_t* src = ev_src + (size_t)b * E_max;
    const Decay* d = dec + (size_t)b * E_pad;
    float* st = out_t + idx * (size_t)m.s_max;
    float* si = out_i ? out_i + idx * (size_t)m.s_max : nullptr;
    int32_t* sk = out_k ? out_k + idx * (size_t)m.s_max : nullptr;
    int ns = 0;
    bool capped = false;
    double V = 0.0, I = 0.0, t_prev = 0.0;
    for (int k = 0; k <= nb && !capped; ++k) {
        double L, A, C, Dd;
        if (k < nb) {
            Decay e = d[k];
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
            I = Dd * I + (double)WT[(size_t)clamp_src(src[k], C_in) * (size_t)N + n];
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
    L.agg = take(BS * N * sizeof(double2));
    L.carry = take(BS * N * sizeof(double2));
    L.mask = take(BS * N * sizeof(uint2));
    L.ent = take(BS * kSubPerSeg * N * sizeof(double2));
    // per sample: record-pool use, work-list length
    L.n_counters = 2 * (size_t)B * kCtr;
    L.counters = take(L.n_counters * sizeof(uint32_t));
    L.listed = take((size_t)B * N * sizeof(uint32_t));
    L.work = take((size_t)B * N * sizeof(uint32_t));
    // Record pool: one record per flagged (sub-block, neuron), in per-sample
    // slices sized at a 16th of the dense bound (every sub-block of every
    // neuron flagged), at least 4096 records (or the dense bound when
    // smaller).  A full slice only sends the excess sub-blocks through a
    // slower re-walk.  lif_params.pool_cap >= 0 sets the slice size (tests
    // of the re-walk path).
    const size_t dense = (size_t)L.S * kSubPerSeg * N;
    size_t cap = dense / 16 > 4096 ? dense / 16 : (dense < 4096 ? dense : 4096);
    if (pool_cap >= 0) cap = (size_t)pool_cap;
    if (B > 0 && (size_t)B * cap > 0xfffffff0ull) cap = 0xfffffff0ull / (size_t)B;   // slot indices are 32-bit
    L.pool_cap = cap;
    const size_t recs = (size_t)B * cap;
    L.pool = take((recs > 0 ? recs : 1) * sizeof(Record));   // at least one record (a safe load address)
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
    double2 *segm, *agg, *carry, *ent;
    uint2* mask;
    uint32_t *counters, *pool_count, *nwork, *listed, *work;
    Record* pool;
};

template <int NPL>
static void launch_walks(const FwdLayout& L, const FwdPtrs& P, const float* ev_t, const int32_t* ev_src,
                         const int32_t* ev_n, int B, int E_max, const float* WT, int C_in, int N, const Model& m,
                         int32_t* status, bool validate, hipStream_t stream)
{
    const int tiles = (N + kWave * NPL - 1) / (kWave * NPL);
    const size_t items = (size_t)B * L.S * tiles;
    const unsigned blocks = (unsigned)((items + kWalkWaves - 1) / kWalkWaves);
    // the aggregate pass also computes the decays and resets the counters and
    // status words (validation flags are ORed in after it)
    TIMED_LAUNCH("aggregate", k_aggregate<NPL>, dim3(blocks), dim3(kWave * kWalkWaves), 0, stream,
                 ev_t, ev_src, ev_n, E_max, L.E_pad, WT, C_in, N, tiles, L.S, (int)items, m, P.dec, P.segm, P.agg,
                 status, P.counters, L.n_counters, P.listed, (size_t)B * N);
    if (validate)
        TIMED_LAUNCH("validate", k_validate, dim3((unsigned)(((size_t)B * E_max + 255) / 256)), dim3(256), 0,
                     stream, ev_t, ev_src, ev_n, B, E_max, C_in, status);
    const int ctiles = (N + kWave - 1) / kWave;
    TIMED_LAUNCH("carry", k_carry, dim3((unsigned)((size_t)B * ctiles)), dim3(kWave * kCarryWaves), 0, stream,
                 ev_n, B, E_max, N, ctiles, L.S, P.segm, P.agg, P.carry);
    // The check pass takes one neuron per lane whatever NPL the aggregate
    // uses: its screen and record state make wider lanes cost occupancy
    // (about 200 VGPRs at four neurons per lane against under 80 at one).
    const int ctl = (N + kWave - 1) / kWave;
    const size_t citems = (size_t)B * L.S * ctl;
    const unsigned cblocks = (unsigned)((citems + kWalkWaves - 1) / kWalkWaves);
    TIMED_LAUNCH("check", k_check, dim3(cblocks), dim3(kWave * kWalkWaves), 0, stream,
                 ev_t, ev_src, ev_n, E_max, L.E_pad, WT, C_in, N, ctl, L.S, (int)citems, m, P.dec, P.carry, P.ent,
                 P.mask, P.pool, P.pool_count, (uint32_t)L.pool_cap, P.listed, P.work, P.nwork);
}

int forward_impl(bool sequential, const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                 const float* WT, int C_in, int N, const lif_params* p, float* out_t, int32_t* out_n,
                 float* out_i, int32_t* out_k, int32_t* status, void* ws, size_t ws_bytes, hipStream_t stream)
{
    int rc = validate_forward_args(ev_t, ev_src, ev_n, B, E_max, WT, C_in, N, p, out_t, out_n, status, ws);
    if (rc) return rc;
    FwdLayout L = fwd_layout(B, E_max, N, p->pool_cap);
    if (ws_bytes < L.total) return LIF_ERR_WORKSPACE;
    Model m = make_model(*p);
    char* base = (char*)(((uintptr_t)ws + 255) & ~(uintptr_t)255);
    FwdPtrs P;
    P.dec = (Decay*)(base + L.dec);
    P.segm = (double2*)(base + L.segm);
    P.agg = (double2*)(base + L.agg);
    P.carry = (double2*)(base + L.carry);
    P.ent = (double2*)(base + L.ent);
    P.mask = (uint2*)(base + L.mask);
    P.counters = (uint32_t*)(base + L.counters);
    P.pool_count = P.counters;
    P.nwork = P.counters + (size_t)B * kCtr;
    P.listed = (uint32_t*)(base + L.listed);
    P.work = (uint32_t*)(base + L.work);
    P.pool = (Record*)(base + L.pool);

    const size_t nev = (size_t)B * L.E_pad;
    const size_t nn = (size_t)B * N;
    const size_t items_max = (size_t)B * L.S * ((N + kWave - 1) / kWave);
    if (items_max > 0x7fffffff || nn > 0xffffffffull) return LIF_ERR_SIZE;
    const size_t n_out = nn * (size_t)p->s_max;
    const bool validate = (p->flags & LIF_VALIDATE) && (size_t)B * E_max;
    if (sequential || items_max == 0) {
        // decays and resets in their own pass (the parallel path folds them
        // into the aggregate and record passes)
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
            TIMED_LAUNCH("sequential", k_sequential, dim3((unsigned)((nn + 63) / 64)), dim3(64), 0, stream,
                         ev_t, ev_src, ev_n, B, E_max, WT, C_in, N, m, L.E_pad, P.dec, out_t, out_n, out_i, out_k);
        TIMED_LAUNCH("status", k_status, dim3(status_blocks(B, N)), dim3(kStatusThreads), 0, stream, ev_n, B, E_max, N, m.s_max, out_n,
                     status);
        return check_launch();
    }
    if (items_max == 0) return check_launch();
    switch (pick_npl(WT, N)) {
    case 4: launch_walks<4>(L, P, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N, m, status, validate, stream); break;
    case 2: launch_walks<2>(L, P, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N, m, status, validate, stream); break;
    default: launch_walks<1>(L, P, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N, m, status, validate, stream); break;
    }
    {
        // 16 blocks of 4 waves per sample (256 records per round), fewer
        // when the pool slice is smaller; the blocks loop over the records
        const size_t per = (L.pool_cap + 15) / 16;
        const unsigned bx = (unsigned)(per < 1 ? 1 : (per > 16 ? 16 : per));
        if (B > 0)
            TIMED_LAUNCH("records", k_records, dim3(bx, (unsigned)B), dim3(256), 0, stream,
                         ev_t, ev_src, ev_n, E_max, L.E_pad, L.S, WT, C_in, N, m, P.dec, P.ent, P.pool, P.pool_count,
                         (uint32_t)L.pool_cap, out_n, nn, out_t, out_i, out_k, n_out, B, status);
    }
    // Two-wave workgroups (chain and staging waves) over the concatenated
    // per-sample lists.
    const unsigned rgrid = (unsigned)(nn < 4096 ? nn : 4096);
    TIMED_LAUNCH("resolve", k_resolve, dim3(rgrid), dim3(kWave * kResolveWaves), 0, stream,
                 ev_t, ev_src, ev_n, B, E_max, WT, C_in, N, L.E_pad, L.S, m, P.dec, P.ent, P.mask, (uint32_t)L.pool_cap,
                 P.pool, P.work, P.nwork, out_t, out_n, out_i, out_k, status);
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
