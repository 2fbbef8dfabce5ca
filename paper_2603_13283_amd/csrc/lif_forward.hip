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

// Record of one flagged sub-block of one neuron: the no-reset state (V, I)
// entering it and right after each of its kSub events.  With the reset
// deficit of the spikes found so far, these give the true state at every
// interval boundary of the sub-block in O(1), so the resolve pass can test
// all of its intervals at once.  Records live in a pool; each wave allocates
// the records of one sub-block with one atomic and notes (lane mask, first
// slot).
struct alignas(16) Record {
    double2 s[kSub + 1];    // s[0]: entering state; s[j + 1]: after event j
};
static_assert(sizeof(Record) == 16 * (kSub + 1), "record layout");

struct alignas(16) WaveInfo {
    unsigned long long lanes;   // lanes of the wave with a record for this sub-block
    uint32_t base;              // pool slot of the lowest such lane, kNoSlot if the pool was full
    uint32_t pad;
};
constexpr uint32_t kNoSlot = 0xffffffffu;

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
// Decay record of event k (gap to the previous event, or to t = 0).
__device__ __forceinline__ Decay make_decay(const Model& m, const float* __restrict__ t, int k)
{
    double dt = (double)t[k] - (k > 0 ? (double)t[k - 1] : 0.0);
    Decay d;
    d.A = exp(-dt * m.inv_tm);
    d.D = exp(-dt * m.inv_ts);
    d.C = unit_kernel(m, dt, d.A);
    double gl = fmin(dt, m.t_peak);
    d.g = unit_kernel(m, gl, exp(-gl * m.inv_tm)) * (1.0 + 1e-12);
    return d;
}

__global__ __launch_bounds__(256) void k_decay(const float* __restrict__ ev_t, const int32_t* __restrict__ ev_n,
                                               int B, int E_max, int S, Model m, Decay* __restrict__ dec,
                                               int32_t* __restrict__ status, uint32_t* __restrict__ counters,
                                               float* __restrict__ out_t, float* __restrict__ out_i, size_t n_out)
{
    const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    if (tid < LIF_STATUS_WORDS) status[tid] = 0;
    if (out_t) {
        for (size_t i = tid; i < n_out; i += stride) {
            out_t[i] = INFINITY;
            if (out_i) out_i[i] = 0.0f;
        }
    }
    const size_t nev = (size_t)B * (size_t)E_max;
    for (size_t idx = tid; idx < nev; idx += stride) {
        int b = (int)(idx / (size_t)E_max), k = (int)(idx % (size_t)E_max);
        if (k >= clamp_count(ev_n[b], E_max)) continue;
        dec[idx] = make_decay(m, ev_t + (size_t)b * E_max, k);
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
// Segment walks.  A workgroup of kTilesPerBlock waves takes one (sample,
// segment) and kTilesPerBlock 64-neuron tiles; lanes are neurons.  The
// segment's decay records are computed (k_aggregate) or fetched (k_check)
// once into LDS and read by all of its waves.  Each event's source is
// wave-uniform; lane j holds the sources of events j and j + 64 and each is
// broadcast with a lane read, so the weight loads of the next kSub events
// (one coalesced W^T row slice per event) are issued while the current kSub
// events are walked.
// ---------------------------------------------------------------------------
constexpr int kTilesPerBlock = 4;
constexpr int kSrcRegs = kSeg / kWave;

struct SegCoords {
    int b, seg, tile, wave, lane, n, nc, nb, k0, cnt;
};

__device__ __forceinline__ SegCoords seg_coords(int total, int tgroups, int S, const int32_t* __restrict__ ev_n,
                                                int E_max, int N)
{
    SegCoords c;
    int lin = xcd_remap(blockIdx.x, total);
    int tg = lin % tgroups;
    int rest = lin / tgroups;
    c.seg = rest % S;
    c.b = rest / S;
    c.wave = (int)threadIdx.x / kWave;
    c.lane = (int)threadIdx.x % kWave;
    c.tile = tg * kTilesPerBlock + c.wave;
    c.n = c.tile * kWave + c.lane;
    c.nc = min(c.n, N - 1);
    c.nb = clamp_count(ev_n[c.b], E_max);
    c.k0 = c.seg * kSeg;
    c.cnt = min(kSeg, c.nb - c.k0);
    return c;
}

struct SrcRegs {
    int v[kSrcRegs];
};

__device__ __forceinline__ SrcRegs load_sources(const int32_t* __restrict__ src, int cnt, int lane, int C_in)
{
    SrcRegs r;
#pragma unroll
    for (int h = 0; h < kSrcRegs; ++h) r.v[h] = h * kWave + lane < cnt ? clamp_src(src[h * kWave + lane], C_in) : 0;
    return r;
}

// Weights of events q*kSub .. q*kSub + kSub - 1 of the segment (0 past cnt).
__device__ __forceinline__ void load_sub_weights(const SrcRegs& sr, const float* __restrict__ wcol, int N, int cnt,
                                                 int q, float (&w)[kSub])
{
#pragma unroll
    for (int j = 0; j < kSub; ++j) {
        const int e = q * kSub + j;
        int sj = __builtin_amdgcn_readlane(sr.v[e / kWave], e % kWave);
        w[j] = e < cnt ? wcol[(size_t)sj * (size_t)N] : 0.0f;
    }
}

__global__ __launch_bounds__(kWave * kTilesPerBlock) void k_aggregate(
    const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src, const int32_t* __restrict__ ev_n, int E_max,
    const float* __restrict__ WT, int C_in, int N, int tiles, int tgroups, int S, int total, Model m,
    Decay* __restrict__ dec, Decay* __restrict__ segm, double2* __restrict__ agg, int32_t* __restrict__ status,
    uint32_t* __restrict__ counters, float* __restrict__ out_t, float* __restrict__ out_i, size_t n_out)
{
    __shared__ Decay sd[kSeg];
    if (blockIdx.x == 0 && threadIdx.x < LIF_STATUS_WORDS) status[threadIdx.x] = 0;
    {
        // Every neuron starts with no spike (+inf times); the resolve pass
        // overwrites the outputs of neurons that fire.  Coalesced fill spread
        // over the whole launch.
        const size_t stride = (size_t)gridDim.x * blockDim.x;
        for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_out; i += stride) {
            out_t[i] = INFINITY;
            if (out_i) out_i[i] = 0.0f;
        }
    }
    const SegCoords c = seg_coords(total, tgroups, S, ev_n, E_max, N);
    if (c.k0 >= c.nb) return;                        // uniform over the workgroup
    const float* tt = ev_t + (size_t)c.b * E_max;
    const int tg = c.tile / kTilesPerBlock;
    if ((int)threadIdx.x < c.cnt) {
        int k = c.k0 + (int)threadIdx.x;
        Decay e = make_decay(m, tt, k);
        sd[threadIdx.x] = e;
        if (tg == 0) dec[(size_t)c.b * E_max + k] = e;
    }
    if (tg == 0 && threadIdx.x == kSeg % (kWave * kTilesPerBlock)) {
        // The segment's composed map M(T) (the maps form a semigroup).
        double T = (double)tt[c.k0 + c.cnt - 1] - (c.k0 > 0 ? (double)tt[c.k0 - 1] : 0.0);
        Decay sm;
        sm.A = exp(-T * m.inv_tm);
        sm.D = exp(-T * m.inv_ts);
        sm.C = unit_kernel(m, T, sm.A);
        sm.g = T;
        segm[(size_t)c.b * S + c.seg] = sm;
    }
    __syncthreads();
    if (c.tile >= tiles) return;
    const float* wcol = WT + c.nc;
    const SrcRegs sr = load_sources(ev_src + (size_t)c.b * E_max + c.k0, c.cnt, c.lane, C_in);
    double V = 0.0, I = 0.0;
    float wn[kSub], wn2[kSub];
    load_sub_weights(sr, wcol, N, c.cnt, 0, wn);
    if (kSub < c.cnt) load_sub_weights(sr, wcol, N, c.cnt, 1, wn2);
#pragma unroll
    for (int q = 0; q < kSubPerSeg; ++q) {
        if (q * kSub < c.cnt) {
            float w[kSub];
#pragma unroll
            for (int j = 0; j < kSub; ++j) { w[j] = wn[j]; wn[j] = wn2[j]; }
            if (q + 2 < kSubPerSeg && (q + 2) * kSub < c.cnt) load_sub_weights(sr, wcol, N, c.cnt, q + 2, wn2);
            if ((q + 1) * kSub <= c.cnt) {            // full sub-block: straight-line code
#pragma unroll
                for (int j = 0; j < kSub; ++j) {
                    Decay e = sd[q * kSub + j];
                    double Vn = e.A * V + e.C * I;
                    I = e.D * I + (double)w[j];
                    V = Vn;
                }
            } else {
                for (int j = 0; j < c.cnt - q * kSub; ++j) {
                    Decay e = sd[q * kSub + j];
                    double Vn = e.A * V + e.C * I;
                    I = e.D * I + (double)w[j];
                    V = Vn;
                }
            }
        }
    }
    if (c.n < N) agg[((size_t)c.b * S + c.seg) * N + c.n] = make_double2(V, I);
}

// Exclusive scan over segments of the Combine of Eq. affine:
// s_in(j+1) = M(T_j) s_in(j) + b_j, with s_in(0) = (0, 0).  The segment
// aggregates are fetched kCarryBatch at a time so their loads overlap.
constexpr int kCarryBatch = 16;

__global__ __launch_bounds__(64) void k_carry(const int32_t* __restrict__ ev_n, int B, int E_max, int N, int S,
                                               const Decay* __restrict__ segm, const double2* __restrict__ agg,
                                               double2* __restrict__ carry, int32_t* __restrict__ status,
                                               int s_max, float* __restrict__ out_t, int32_t* __restrict__ out_n,
                                               float* __restrict__ out_i, uint32_t* __restrict__ listed,
                                               uint32_t* __restrict__ counters)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t nn = (size_t)B * (size_t)N;
    if (idx >= nn) return;
    int b = (int)(idx / (size_t)N), n = (int)(idx % (size_t)N);
    out_n[idx] = 0;
    listed[idx] = 0u;
    if (n == 0) counters[1 + b] = 0u;          // record pool use of sample b
    if (idx == 0) counters[0] = 0u;            // work-list length
    int nb = clamp_count(ev_n[b], E_max);
    if (n == 0) atomicAdd(&status[LIF_ST_EVENTS], nb);
    int Sb = (nb + kSeg - 1) / kSeg;
    double V = 0.0, I = 0.0;
    for (int j0 = 0; j0 < Sb; j0 += kCarryBatch) {
        double2 a[kCarryBatch];
#pragma unroll
        for (int j = 0; j < kCarryBatch; ++j) {
            int jj = min(j0 + j, Sb - 1);
            a[j] = agg[((size_t)b * S + jj) * N + n];
        }
#pragma unroll
        for (int j = 0; j < kCarryBatch; ++j) {
            if (j0 + j < Sb) {
                Decay M = segm[(size_t)b * S + j0 + j];
                carry[((size_t)b * S + j0 + j) * N + n] = make_double2(V, I);
                double Vn = M.A * V + M.C * I + a[j].x;
                I = M.D * I + a[j].y;
                V = Vn;
            }
        }
    }
}

// Re-walk from the carried no-reset state with a cheap exact bound per
// interval: V(t) = V0 e^{-t/tm} + I0 K(t) <= max(V0, 0) + max(I0, 0)
// K(min(dt, t_peak)) since 0 <= K(t) <= K(min(dt, t_peak)) on [0, dt].
// Resets only lower V (each is the subtraction of a positive decaying
// term), so a sub-block whose no-reset bound stays below the threshold holds
// no spike whatever happened before it.  Sub-blocks whose bound reaches it
// get a record for the resolve pass, which applies the exact interval rule.
__global__ __launch_bounds__(kWave * kTilesPerBlock) void k_check(
    const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src, const int32_t* __restrict__ ev_n, int E_max,
    const float* __restrict__ WT, int C_in, int N, int tiles, int tgroups, int S, int total, Model m,
    const Decay* __restrict__ dec, const double2* __restrict__ carry, uint32_t* __restrict__ mask,
    WaveInfo* __restrict__ winfo, Record* __restrict__ pool, double* __restrict__ pool_ub,
    uint32_t* __restrict__ pool_count, uint32_t pool_cap, uint32_t* __restrict__ listed, uint32_t* __restrict__ work,
    uint32_t* __restrict__ nwork, int32_t* __restrict__ status)
{
    __shared__ Decay sd[kSeg];
    const SegCoords c = seg_coords(total, tgroups, S, ev_n, E_max, N);
    if (c.k0 >= c.nb) return;                        // uniform over the workgroup
    const float* tt = ev_t + (size_t)c.b * E_max;
    if ((int)threadIdx.x < c.cnt) sd[threadIdx.x] = dec[(size_t)c.b * E_max + c.k0 + threadIdx.x];
    __syncthreads();
    if (c.tile >= tiles) return;
    const int lane = c.lane, n = c.n, nb = c.nb, k0 = c.k0, cnt_seg = c.cnt;
    const float* wcol = WT + c.nc;
    const SrcRegs sr = load_sources(ev_src + (size_t)c.b * E_max + k0, cnt_seg, lane, C_in);
    const size_t row = ((size_t)c.b * S + c.seg) * N;
    double2 c0 = carry[row + c.nc];
    double V = c0.x, I = c0.y;
    uint32_t msk = 0;
    int ncand = 0;
    const unsigned long long below = (1ull << lane) - 1ull;
    float wn[kSub], wn2[kSub];
    load_sub_weights(sr, wcol, N, cnt_seg, 0, wn);
    if (kSub < cnt_seg) load_sub_weights(sr, wcol, N, cnt_seg, 1, wn2);
#pragma unroll
    for (int q = 0; q < kSubPerSeg; ++q) {
        if (q * kSub < cnt_seg) {
            const int cnt = min(kSub, cnt_seg - q * kSub);
            float w[kSub];
#pragma unroll
            for (int j = 0; j < kSub; ++j) { w[j] = wn[j]; wn[j] = wn2[j]; }
            if (q + 2 < kSubPerSeg && (q + 2) * kSub < cnt_seg) load_sub_weights(sr, wcol, N, cnt_seg, q + 2, wn2);
            double Vin = V, Iin = I, ub = -INFINITY;
            if (cnt == kSub) {                         // full sub-block: straight-line code
#pragma unroll
                for (int j = 0; j < kSub; ++j) {
                    Decay e = sd[q * kSub + j];
                    ub = fmax(ub, fmax(V, 0.0) + fmax(I, 0.0) * e.g);
                    double Vn = e.A * V + e.C * I;
                    I = e.D * I + (double)w[j];
                    V = Vn;
                }
            } else {
                for (int j = 0; j < cnt; ++j) {
                    Decay e = sd[q * kSub + j];
                    ub = fmax(ub, fmax(V, 0.0) + fmax(I, 0.0) * e.g);
                    double Vn = e.A * V + e.C * I;
                    I = e.D * I + (double)w[j];
                    V = Vn;
                }
            }
            if (k0 + q * kSub + cnt == nb) {
                // Interval after the last event, up to t_end (default +inf).
                double len = m.t_end - (double)tt[nb - 1];
                if (len > 0.0) {
                    double gl = fmin(len, m.t_peak);
                    double g = unit_kernel(m, gl, exp(-gl * m.inv_tm)) * (1.0 + 1e-12);
                    ub = fmax(ub, fmax(V, 0.0) + fmax(I, 0.0) * g);
                }
            }
            bool surv = ub >= m.th_lo && n < N;
            unsigned long long lanes = __ballot(surv);
            if (lanes) {
                int cntl = __popcll(lanes);
                // Records of sample b live in their own slice of the pool, so
                // the allocation atomics of different samples do not contend.
                uint32_t base = 0;
                if (lane == 0) base = atomicAdd(&pool_count[c.b], (uint32_t)cntl);
                base = __shfl(base, 0, kWave);
                bool ok = (unsigned long long)base + (unsigned long long)cntl <= (unsigned long long)pool_cap;
                base += (uint32_t)c.b * pool_cap;
                if (lane == 0) {
                    WaveInfo wi;
                    wi.lanes = lanes;
                    wi.base = ok ? base : kNoSlot;
                    wi.pad = 0;
                    winfo[(((size_t)c.b * S + c.seg) * tiles + c.tile) * kSubPerSeg + q] = wi;
                }
                if (surv) {
                    if (ok) {
                        // Re-walk the sub-block to store its states.
                        uint32_t slot = base + (uint32_t)__popcll(lanes & below);
                        pool_ub[slot] = ub;
                        Record* r = pool + slot;
                        r->s[0] = make_double2(Vin, Iin);
                        double Vr = Vin, Ir = Iin;
#pragma unroll
                        for (int j = 0; j < kSub; ++j) {
                            if (j < cnt) {
                                Decay e = sd[q * kSub + j];
                                double Vn = e.A * Vr + e.C * Ir;
                                Ir = e.D * Ir + (double)w[j];
                                Vr = Vn;
                            }
                            r->s[j + 1] = make_double2(Vr, Ir);
                        }
                    }
                    msk |= 1u << q;
                    ++ncand;
                }
            }
        }
    }
    if (n < N) {
        mask[row + n] = msk;
        if (ncand) {
            size_t bn = (size_t)c.b * N + n;
            if (atomicOr(&listed[bn], 1u) == 0u) work[atomicAdd(nwork, 1u)] = (uint32_t)bn;
        }
    }
    int tot = ncand;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) tot += __shfl_xor(tot, off, kWave);
    if (lane == 0 && tot) atomicAdd(&status[LIF_ST_CAND_BLOCKS], tot);
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
        // Decays of the whole gap from the table while no spike split it;
        // after a spike (or for the open last interval) they are computed
        // and the cheap bound is skipped (the exact rule is applied).
        double eA, eD, C;
        bool test = true;
        if (fresh) {
            eA = tab->A; eD = tab->D; C = tab->C;
            test = fmax(V, 0.0) + fmax(I, 0.0) * tab->g >= m.th_lo;
        } else if (isinf(len)) {
            eA = 0.0; eD = 0.0; C = 0.0;
        } else {
            eA = exp(-len * m.inv_tm);
            eD = exp(-len * m.inv_ts);
            C = m.kappa * (eA - eD);
        }
        double vend = V * eA + C * I;
        if (test) {
            Crossing c = interval_rule(m, V, I, len, eA, eD, vend, m.th);
            if (c.hit) {
                int it = 0;
                double tau = newton_root(m, V, I, c.hi, c.vhi, &it);
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

// Rebuild a sub-block's entering no-reset state from its segment carry by
// walking the earlier sub-blocks of the segment (used only when the record
// pool was full).
__device__ __noinline__ double2 entering_state(const double2* __restrict__ carry, size_t row, int n, int k0, int kq0,
                                               const int32_t* __restrict__ src, const Decay* __restrict__ d,
                                               const float* __restrict__ WT, int C_in, int N)
{
    double2 c = carry[row + n];
    double V = c.x, I = c.y;
    for (int k = k0; k < kq0; ++k) {
        Decay e = d[k];
        double Vn = e.A * V + e.C * I;
        I = e.D * I + (double)WT[(size_t)clamp_src(src[k], C_in) * (size_t)N + n];
        V = Vn;
    }
    return make_double2(V, I);
}

// Resolve pass: one wave per neuron that has flagged sub-blocks (a work
// list built by the check pass); the paper's chunked speculative scheme
// applied to those sub-blocks only.
//   * Flagged sub-blocks are taken in time order in windows of kWin.  A
//     window's records (no-reset states), decays and event times are staged
//     in LDS with one batch of loads (one lane per sub-block).
//   * Since every reset subtracts (V_th - V_reset) e^{-(t - t_s)/tm} from
//     the no-reset trajectory, the true state entering an interval is the
//     record's no-reset state minus the reset deficit at its start.  A
//     sub-block whose no-reset bound minus the deficit at its end stays
//     below the threshold is certified at once (more spikes only deepen the
//     deficit); this test runs for the whole window in parallel.
//   * The earliest kGroup uncertified sub-blocks are checked together, one
//     lane per interval, with the interval rule; the earliest crossing
//     (ballot) is solved by its lane with bracketed Newton, reset and
//     re-tested until its interval is clear, the deficit is updated and the
//     later intervals are tested again.
// Intervals outside flagged sub-blocks provably hold no spike.
constexpr int kGroup = kWave / kSub;
constexpr int kWin = 32;

// Wave-uniform spike bookkeeping of the neuron being resolved.
struct NeuronSpikes {
    int ns, roots;
    double dref, tref;    // reset deficit dref at time tref
    bool capped;
};

__device__ __forceinline__ double deficit_at(const NeuronSpikes& ns_, const Model& m, double t)
{
    return ns_.ns > 0 ? ns_.dref * exp(-(t - ns_.tref) * m.inv_tm) : 0.0;
}

__device__ __forceinline__ void share_from(NeuronSpikes& sp, int from)
{
    sp.ns = __shfl(sp.ns, from, kWave);
    sp.roots = __shfl(sp.roots, from, kWave);
    sp.dref = __shfl(sp.dref, from, kWave);
    sp.tref = __shfl(sp.tref, from, kWave);
    sp.capped = __shfl((int)sp.capped, from, kWave) != 0;
}

struct ResolveLds {
    double2 s[kWin][kSub + 1];   // no-reset states: entering, then after each event
    Decay e[kWin][kSub];         // decays of the sub-block's events
    float t[kWin][kSub + 1];     // time before the sub-block, then each event's time
    int seg[kWin], q[kWin];      // the window's sub-blocks
    int grp[kGroup];             // window slots of the group being checked
};

__device__ void resolve_neuron(ResolveLds& sh, int b, int n, const float* __restrict__ ev_t,
                               const int32_t* __restrict__ ev_src, const int32_t* __restrict__ ev_n, int E_max,
                               const float* __restrict__ WT, int C_in, int N, int tiles, int S, const Model& m,
                               const Decay* __restrict__ dec, const double2* __restrict__ carry,
                               const uint32_t* __restrict__ mask, const WaveInfo* __restrict__ winfo,
                               const Record* __restrict__ pool, const double* __restrict__ pool_ub,
                               float* __restrict__ out_t, int32_t* __restrict__ out_n, float* __restrict__ out_i,
                               int32_t* __restrict__ status)
{
    const int tile = n / kWave;
    const unsigned long long below_n = (1ull << (n % kWave)) - 1ull;
    const int lane = (int)threadIdx.x;
    const int nb = clamp_count(ev_n[b], E_max);
    const float* tt = ev_t + (size_t)b * E_max;
    const int32_t* src = ev_src + (size_t)b * E_max;
    const Decay* d = dec + (size_t)b * E_max;
    const size_t idx = (size_t)b * N + n;
    float* st = out_t + idx * (size_t)m.s_max;
    float* si = out_i ? out_i + idx * (size_t)m.s_max : nullptr;
    NeuronSpikes sp{0, 0, 0.0, 0.0, false};
    int walked = 0, fallback = 0;
    const int Sb = (nb + kSeg - 1) / kSeg;
    int W = 0;

    auto process_window = [&]() {
        __syncthreads();                                  // window list written by lane 0
        // ---- stage: lane c loads sub-block c's record, decays and times
        bool done = lane >= W;
        double ub = 0.0, t_out = 0.0;
        int cnt_c = 0;
        if (!done) {
            int seg = sh.seg[lane], q = sh.q[lane];
            int kq0 = seg * kSeg + q * kSub;
            cnt_c = min(kSub, nb - kq0);
            WaveInfo wi = winfo[(((size_t)b * S + seg) * tiles + tile) * kSubPerSeg + q];
            {
                float tv[kSub + 1];
                Decay ev[kSub];
                tv[0] = kq0 > 0 ? tt[kq0 - 1] : 0.0f;
#pragma unroll
                for (int j = 0; j < kSub; ++j) {
                    int k = min(kq0 + j, nb - 1);
                    ev[j] = d[k];
                    tv[j + 1] = tt[k];
                }
#pragma unroll
                for (int j = 0; j < kSub; ++j) sh.e[lane][j] = ev[j];
#pragma unroll
                for (int j = 0; j <= kSub; ++j) sh.t[lane][j] = tv[j];
            }
            if (wi.base != kNoSlot) {
                uint32_t slot = wi.base + (uint32_t)__popcll(wi.lanes & below_n);
                ub = pool_ub[slot];
                const Record* rec = pool + slot;
                double2 rs[kSub + 1];
#pragma unroll
                for (int j = 0; j <= kSub; ++j) rs[j] = rec->s[j];
#pragma unroll
                for (int j = 0; j <= kSub; ++j) sh.s[lane][j] = rs[j];
            } else {
                size_t row = ((size_t)b * S + seg) * N;
                double2 cs = entering_state(carry, row, n, seg * kSeg, kq0, src, d, WT, C_in, N);
                double V = cs.x, I = cs.y;
                sh.s[lane][0] = cs;
                for (int j = 0; j < kSub; ++j) {
                    if (j < cnt_c) {
                        Decay e = d[kq0 + j];
                        double Vn = e.A * V + e.C * I;
                        I = e.D * I + (double)WT[(size_t)clamp_src(src[kq0 + j], C_in) * (size_t)N + n];
                        V = Vn;
                    }
                    sh.s[lane][j + 1] = make_double2(V, I);
                }
                ub = INFINITY;
            }
            double tl = (double)tt[kq0 + cnt_c - 1];
            t_out = kq0 + cnt_c == nb ? fmax(m.t_end, tl) : tl;
        }
        fallback += __popcll(__ballot(ub == INFINITY && lane < W));
        __syncthreads();
        // Deficits are evaluated as dw * e^{-(t - tw)/tm}: the per-lane factor
        // is computed once per window (or group), the uniform dw only after
        // a spike.
        const double tw = (double)sh.t[0][0];
        const double f_out = isinf(t_out) ? 0.0 : exp(-(t_out - tw) * m.inv_tm);
        double dw = deficit_at(sp, m, tw);
        int dw_ns = sp.ns;
        while (!sp.capped) {
            if (sp.ns != dw_ns) { dw = deficit_at(sp, m, tw); dw_ns = sp.ns; }
            // ---- certify in parallel with the current deficit
            if (!done && sp.ns > 0) {
                if (ub - dw * f_out < m.th_lo) done = true;
            }
            unsigned long long rem = __ballot(!done);
            if (!rem) break;
            // ---- the earliest kGroup uncertified sub-blocks form the group
            int G = 0;
            while (rem && G < kGroup) {
                int c = __ffsll((long long)rem) - 1;
                rem &= rem - 1ull;
                if (lane == 0) sh.grp[G] = c;
                if (lane == c) done = true;
                ++G;
            }
            __syncthreads();
            walked += G;
            const int r = lane / kSub, j = lane % kSub;
            const int c = r < G ? sh.grp[r] : 0;
            int kq0 = 0, cnt = 0;
            if (r < G) { kq0 = sh.seg[c] * kSeg + sh.q[c] * kSub; cnt = min(kSub, nb - kq0); }
            const bool valid = r < G && j < cnt;
            const Decay e = valid ? sh.e[c][j] : Decay{1.0, 0.0, 1.0, 0.0};
            const double t0 = valid ? (double)sh.t[c][j] : 0.0;
            const double t1 = valid ? (double)sh.t[c][j + 1] : 0.0;
            const double2 s0 = valid ? sh.s[c][j] : make_double2(0.0, 0.0);
            const double2 s1 = valid ? sh.s[c][j + 1] : make_double2(0.0, 0.0);
            bool pending = valid && t1 > t0;
            const double f0 = exp(-(t0 - tw) * m.inv_tm);
            while (!sp.capped) {
                if (sp.ns != dw_ns) { dw = deficit_at(sp, m, tw); dw_ns = sp.ns; }
                bool cross = false;
                double V0 = 0.0, I0 = 0.0;
                if (pending) {
                    double def0 = dw * f0;
                    V0 = s0.x - def0;
                    I0 = s0.y;
                    double u = fmax(V0, 0.0) + fmax(I0, 0.0) * e.g;
                    if (u >= m.th_lo) cross = interval_rule(m, V0, I0, t1 - t0, e.A, e.D, s1.x - def0 * e.A, m.th).hit;
                }
                unsigned long long cm = __ballot(cross);
                if (!cm) break;
                const int kl = __ffsll((long long)cm) - 1;
                if (lane == kl) {
                    Sink sk;
                    sk.st = st; sk.si = si;
                    sk.ns = sp.ns; sk.roots = sp.roots; sk.dref = sp.dref; sk.tref = sp.tref;
                    double V = V0, I = I0, tc = t0;
                    bool ok = advance_interval(m, V, I, tc, t1, &e, sk);
                    sp.ns = sk.ns; sp.roots = sk.roots; sp.dref = sk.dref; sp.tref = sk.tref;
                    sp.capped = !ok;
                }
                share_from(sp, kl);
                if (lane <= kl) pending = false;
            }
            // ---- the open interval after the stream's last event
            if (!sp.capped) {
                const int cl = sh.grp[G - 1];
                int kql = sh.seg[cl] * kSeg + sh.q[cl] * kSub;
                int cntl = min(kSub, nb - kql);
                if (kql + cntl == nb) {
                    if (lane == 0) {
                        double tl = (double)sh.t[cl][cntl];
                        double2 sl = sh.s[cl][cntl];
                        Sink sk;
                        sk.st = st; sk.si = si;
                        sk.ns = sp.ns; sk.roots = sp.roots; sk.dref = sp.dref; sk.tref = sp.tref;
                        double V = sl.x - deficit_at(sp, m, tl), I = sl.y, tc = tl;
                        bool ok = advance_interval(m, V, I, tc, m.t_end, nullptr, sk);
                        sp.ns = sk.ns; sp.roots = sk.roots; sp.dref = sk.dref; sp.tref = sk.tref;
                        sp.capped = !ok;
                    }
                    share_from(sp, 0);
                }
            }
            __syncthreads();
        }
        __syncthreads();
        W = 0;
    };

    for (int seg0 = 0; seg0 < Sb && !sp.capped; seg0 += kWave) {
        int sj = seg0 + lane;
        uint32_t mv = sj < Sb ? mask[((size_t)b * S + sj) * N + n] : 0u;
        unsigned long long nz = __ballot(mv != 0u);
        while (nz && !sp.capped) {
            int l = __ffsll((long long)nz) - 1;
            nz &= nz - 1ull;
            uint32_t mm = (uint32_t)__shfl((int)mv, l, kWave);
            while (mm && !sp.capped) {
                int q = __builtin_ctz(mm);
                mm &= mm - 1u;
                if (lane == 0) { sh.seg[W] = seg0 + l; sh.q[W] = q; }
                ++W;
                if (W == kWin) process_window();
            }
        }
    }
    if (W > 0 && !sp.capped) process_window();

    if (lane == 0) {
        if (walked) atomicAdd(&status[LIF_ST_WALKED_BLOCKS], walked);
        if (fallback) atomicAdd(&status[LIF_ST_POOL_FALLBACK], fallback);
        out_n[idx] = sp.ns;
        if (sp.capped) {
            atomicAdd(&status[LIF_ST_CAPPED], 1);
            atomicOr(&status[LIF_ST_FLAGS], LIF_WARN_SPIKE_CAP);
        }
        if (sp.ns) atomicAdd(&status[LIF_ST_SPIKES], sp.ns);
        if (sp.roots) atomicAdd(&status[LIF_ST_ROOT_SOLVES], sp.roots);
    }
    __syncthreads();
}

// Work-list driven: every wave takes neurons from the list built by k_check
// until the list is exhausted.
__global__ __launch_bounds__(kWave) void k_resolve(const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src,
                                                   const int32_t* __restrict__ ev_n, int E_max,
                                                   const float* __restrict__ WT, int C_in, int N, int tiles, int S,
                                                   Model m, const Decay* __restrict__ dec,
                                                   const double2* __restrict__ carry,
                                                   const uint32_t* __restrict__ mask,
                                                   const WaveInfo* __restrict__ winfo,
                                                   const Record* __restrict__ pool,
                                                   const double* __restrict__ pool_ub,
                                                   const uint32_t* __restrict__ work, const uint32_t* __restrict__ nwork,
                                                   float* __restrict__ out_t, int32_t* __restrict__ out_n,
                                                   float* __restrict__ out_i, int32_t* __restrict__ status)
{
    __shared__ ResolveLds sh;
    const uint32_t count = *nwork;
    for (uint32_t w = blockIdx.x; w < count; w += gridDim.x) {
        uint32_t bn = work[w];
        resolve_neuron(sh, (int)(bn / (uint32_t)N), (int)(bn % (uint32_t)N), ev_t, ev_src, ev_n, E_max, WT, C_in, N,
                       tiles, S, m, dec, carry, mask, winfo, pool, pool_ub, out_t, out_n, out_i, status);
    }
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
    int tiles = (N + kWave - 1) / kWave;
    L.winfo = take((size_t)B * L.S * tiles * kSubPerSeg * sizeof(WaveInfo));
    L.counters = take(((size_t)B + 1) * sizeof(uint32_t));
    L.listed = take((size_t)B * N * sizeof(uint32_t));
    L.work = take((size_t)B * N * sizeof(uint32_t));
    // Record pool: one record per flagged (sub-block, neuron).  Sized at a
    // sixteenth of the dense bound (far above what spiking activity needs); a
    // full pool only sends the excess sub-blocks through a slower re-walk.
    size_t dense = (size_t)B * L.S * kSubPerSeg * N;
    size_t cap = dense / 16 > 65536 ? dense / 16 : (dense < 65536 ? dense : 65536);
    if (const char* env = getenv("LIF_POOL_CAP")) cap = (size_t)strtoull(env, nullptr, 10);
    if (cap > 0xfffffff0ull) cap = 0xfffffff0ull;
    L.pool_cap = cap;
    L.pool = take(cap * sizeof(Record));
    L.pool_ub = take(cap * sizeof(double));
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
    WaveInfo* winfo = (WaveInfo*)(base + L.winfo);
    uint32_t* counters = (uint32_t*)(base + L.counters);
    uint32_t* nwork = counters;
    uint32_t* pool_count = counters + 1;
    uint32_t* listed = (uint32_t*)(base + L.listed);
    uint32_t* work = (uint32_t*)(base + L.work);
    Record* pool = (Record*)(base + L.pool);
    double* pool_ub = (double*)(base + L.pool_ub);

    size_t nev = (size_t)B * E_max;
    size_t nn = (size_t)B * N;
    int tiles = (N + kWave - 1) / kWave;
    int tgroups = (tiles + kTilesPerBlock - 1) / kTilesPerBlock;
    size_t total = (size_t)B * L.S * tgroups;
    if (total > 0x7fffffff || nn > 0xffffffffull) return LIF_ERR_SIZE;
    if (sequential || total == 0) {
        size_t blocks = ((nev > nn * (size_t)p->s_max ? nev : nn * (size_t)p->s_max) + 255) / 256;
        if (blocks > 2048) blocks = 2048;
        if (blocks < 1) blocks = 1;
        TIMED_LAUNCH("decay", k_decay, dim3((unsigned)blocks), dim3(256), 0, stream,
                     ev_t, ev_n, B, E_max, L.S, m, dec, status, counters, sequential ? nullptr : out_t, out_i,
                     nn * (size_t)p->s_max);
    } else {
        TIMED_LAUNCH("aggregate", k_aggregate, dim3((unsigned)total), dim3(kWave * kTilesPerBlock), 0, stream,
                     ev_t, ev_src, ev_n, E_max, WT, C_in, N, tiles, tgroups, L.S, (int)total, m, dec, segm, agg,
                     status, counters, out_t, out_i, nn * (size_t)p->s_max);
    }
    if ((p->flags & LIF_VALIDATE) && nev)
        TIMED_LAUNCH("validate", k_validate, dim3((unsigned)((nev + 255) / 256)), dim3(256), 0, stream,
                     ev_t, ev_src, ev_n, B, E_max, C_in, status);
    if (sequential) {
        TIMED_LAUNCH("sequential", k_sequential, dim3((unsigned)((nn + 63) / 64)), dim3(64), 0, stream,
                     ev_t, ev_src, ev_n, B, E_max, WT, C_in, N, m, dec, out_t, out_n, out_i, status);
        return check_launch();
    }
    if (nn)
        TIMED_LAUNCH("carry", k_carry, dim3((unsigned)((nn + 63) / 64)), dim3(64), 0, stream,
                     ev_n, B, E_max, N, L.S, segm, agg, carry, status, m.s_max, out_t, out_n, out_i, listed,
                     counters);
    if (total) {
        TIMED_LAUNCH("check", k_check, dim3((unsigned)total), dim3(kWave * kTilesPerBlock), 0, stream,
                     ev_t, ev_src, ev_n, E_max, WT, C_in, N, tiles, tgroups, L.S, (int)total, m, dec, carry, mask,
                     winfo, pool, pool_ub, pool_count, (uint32_t)(L.pool_cap / (B > 0 ? B : 1)), listed, work, nwork,
                     status);
        // One wave per listed neuron, as many as can be resident at once.
        unsigned grid = (unsigned)(nn < 4096 ? nn : 4096);
        TIMED_LAUNCH("resolve", k_resolve, dim3(grid), dim3(kWave), 0, stream,
                     ev_t, ev_src, ev_n, E_max, WT, C_in, N, tiles, L.S, m, dec, carry, mask, winfo, pool, pool_ub,
                     work, nwork, out_t, out_n, out_i, status);
    }
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
