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
constexpr int kPoolLocal = 16;     // record slots owned by each check wave
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

// The same, with the sources read as wave-uniform (scalar) loads.  All
// sixteen source loads are issued before the first is used (past cnt the
// last event is read again and its weight discarded).
__device__ __forceinline__ void load_sub_weights_s(const int32_t* __restrict__ sseg, const float* __restrict__ wcol,
                                                   int N, int C_in, int cnt, int q, float (&w)[kSub])
{
    int sj[kSub];
#pragma unroll
    for (int j = 0; j < kSub; ++j) sj[j] = sseg[min(q * kSub + j, cnt - 1)];
#pragma unroll
    for (int j = 0; j < kSub; ++j) w[j] = wcol[(size_t)clamp_src(sj[j], C_in) * (size_t)N];
#pragma unroll
    for (int j = 0; j < kSub; ++j)
        if (q * kSub + j >= cnt) w[j] = 0.0f;
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
// s_in(j+1) = M(T_j) s_in(j) + b_j, with s_in(0) = (0, 0).  A workgroup of
// kCarryWaves waves takes one (sample, 64-neuron tile); lanes are neurons
// and wave w the w-th contiguous range of segments.  Each wave folds its
// range from the zero state (the segment aggregates are fetched
// kCarryBatch at a time so that their loads overlap), the range totals are
// combined across waves in LDS (the maps compose in closed form), and each
// wave walks its range again from its incoming state, writing the carries.
constexpr int kCarryBatch = 16;
constexpr int kCarryWaves = 4;

struct Affine {               // the map s -> M s + b of a range of segments
    double A, C, D;           // M = [[A, C], [0, D]] (wave-uniform)
    double V, I;              // b (per neuron)
};

__device__ __forceinline__ void carry_batch(const double2* __restrict__ agg, const Decay* __restrict__ segm,
                                            size_t row0, size_t seg_row, int N, int n, int j0, int j1,
                                            double2 (&a)[kCarryBatch], double (&mA)[kCarryBatch],
                                            double (&mC)[kCarryBatch], double (&mD)[kCarryBatch])
{
#pragma unroll
    for (int j = 0; j < kCarryBatch; ++j) {
        const int jj = min(j0 + j, j1 - 1);
        a[j] = agg[(row0 + (size_t)jj) * N + n];
        const Decay* M = segm + seg_row + jj;
        mA[j] = __builtin_nontemporal_load(&M->A);
        mC[j] = __builtin_nontemporal_load(&M->C);
        mD[j] = __builtin_nontemporal_load(&M->D);
    }
}

__global__ __launch_bounds__(kWave * kCarryWaves) void k_carry(
    const int32_t* __restrict__ ev_n, int B, int E_max, int N, int tiles, int S, const Decay* __restrict__ segm,
    const double2* __restrict__ agg, double2* __restrict__ carry, int32_t* __restrict__ status,
    int32_t* __restrict__ out_n, uint32_t* __restrict__ listed, uint32_t* __restrict__ counters)
{
    __shared__ Affine tot[kCarryWaves][kWave];
    const int b = blockIdx.x / tiles, tile = blockIdx.x % tiles;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int n = tile * kWave + lane;
    const bool live = n < N;
    const int nc = live ? n : N - 1;
    const size_t idx = (size_t)b * N + nc;
    if (wave == 0 && live) {
        out_n[idx] = 0;
        listed[idx] = 0u;
    }
    const int nb = clamp_count(ev_n[b], E_max);
    if (threadIdx.x == 0 && tile == 0) {
        counters[b] = 0u;                       // record pool use of sample b
        counters[B + b] = 0u;                   // work-list length of sample b
        atomicAdd(&status[LIF_ST_EVENTS], nb);
    }
    const int Sb = (nb + kSeg - 1) / kSeg;
    const int per = (Sb + kCarryWaves - 1) / kCarryWaves;
    const int j_lo = min(wave * per, Sb), j_hi = min(j_lo + per, Sb);
    const size_t row0 = (size_t)b * S, seg_row = (size_t)b * S;

    // ---- fold this wave's range from the zero state
    Affine f{1.0, 0.0, 1.0, 0.0, 0.0};
    double2 a[kCarryBatch];
    double mA[kCarryBatch], mC[kCarryBatch], mD[kCarryBatch];
    for (int j0 = j_lo; j0 < j_hi; j0 += kCarryBatch) {
        carry_batch(agg, segm, row0, seg_row, N, nc, j0, j_hi, a, mA, mC, mD);
#pragma unroll
        for (int j = 0; j < kCarryBatch; ++j) {
            if (j0 + j < j_hi) {
                const double Vn = mA[j] * f.V + mC[j] * f.I + a[j].x;
                f.I = mD[j] * f.I + a[j].y;
                f.V = Vn;
                // M_j composed after the range so far: [[A_j A, A_j C + C_j D], [0, D_j D]]
                const double Cn = mA[j] * f.C + mC[j] * f.D;
                f.A *= mA[j];
                f.D *= mD[j];
                f.C = Cn;
            }
        }
    }
    tot[wave][lane] = f;
    __syncthreads();
    // ---- incoming state: the earlier ranges applied in order to zero
    double V = 0.0, I = 0.0;
    for (int w = 0; w < wave; ++w) {
        const Affine g = tot[w][lane];
        const double Vn = g.A * V + g.C * I + g.V;
        I = g.D * I + g.I;
        V = Vn;
    }
    // ---- walk the range again, writing the carry entering each segment
    for (int j0 = j_lo; j0 < j_hi; j0 += kCarryBatch) {
        carry_batch(agg, segm, row0, seg_row, N, nc, j0, j_hi, a, mA, mC, mD);
#pragma unroll
        for (int j = 0; j < kCarryBatch; ++j) {
            if (j0 + j < j_hi) {
                if (live) carry[(row0 + (size_t)(j0 + j)) * N + n] = make_double2(V, I);
                const double Vn = mA[j] * V + mC[j] * I + a[j].x;
                I = mD[j] * I + a[j].y;
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
__device__ __forceinline__ int B_of(int total, int tgroups, int S) { return total / (tgroups * S); }

__global__ __launch_bounds__(kWave * kTilesPerBlock) void k_check(
    const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src, const int32_t* __restrict__ ev_n, int E_max,
    const float* __restrict__ WT, int C_in, int N, int tiles, int tgroups, int S, int total, Model m,
    const Decay* __restrict__ dec, const double2* __restrict__ carry, double2* __restrict__ ent,
    uint32_t* __restrict__ mask, WaveInfo* __restrict__ winfo, Record* __restrict__ pool,
    uint32_t* __restrict__ pool_count, uint32_t pool_local, uint32_t pool_cap, uint32_t* __restrict__ listed,
    uint32_t* __restrict__ work, uint32_t* __restrict__ nwork, int32_t* __restrict__ status)
// work: per-sample lists of the neurons with candidates (capacity N each);
// nwork: per-sample list lengths.
{
    // The segment's decays and sources are wave-uniform: they are read with
    // scalar loads and used as scalar operands.
    const SegCoords c = seg_coords(total, tgroups, S, ev_n, E_max, N);
    if (c.k0 >= c.nb || c.tile >= tiles) return;
    const float* tt = ev_t + (size_t)c.b * E_max;
    const int lane = c.lane, n = c.n, nb = c.nb, k0 = c.k0, cnt_seg = c.cnt;
    const float* wcol = WT + c.nc;
    const Decay* __restrict__ sd = dec + (size_t)c.b * E_max + k0;
    const int32_t* __restrict__ sseg = ev_src + (size_t)c.b * E_max + k0;
    const size_t row = ((size_t)c.b * S + c.seg) * N;
    double2 c0 = carry[row + c.nc];
    double V = c0.x, I = c0.y;
    uint32_t msk = 0;
    int ncand = 0;
    const unsigned long long below = (1ull << lane) - 1ull;
    // Records go first to this wave's own block of pool_local slots (no
    // atomic), then to the per-sample overflow slices (one atomic each).
    const uint32_t wave_id = (uint32_t)(((size_t)c.b * S + c.seg) * tiles + c.tile);
    const uint32_t local0 = wave_id * pool_local;
    const uint32_t overflow0 = (uint32_t)((size_t)B_of(total, tgroups, S) * S * tiles * pool_local);
    uint32_t used = 0;
    float wn[kSub], wn2[kSub];
    load_sub_weights_s(sseg, wcol, N, C_in, cnt_seg, 0, wn);
    if (kSub < cnt_seg) load_sub_weights_s(sseg, wcol, N, C_in, cnt_seg, 1, wn2);
#pragma unroll
    for (int q = 0; q < kSubPerSeg; ++q) {
        if (q * kSub < cnt_seg) {
            const int cnt = min(kSub, cnt_seg - q * kSub);
            float w[kSub];
#pragma unroll
            for (int j = 0; j < kSub; ++j) { w[j] = wn[j]; wn[j] = wn2[j]; }
            if (q + 2 < kSubPerSeg && (q + 2) * kSub < cnt_seg)
                load_sub_weights_s(sseg, wcol, N, C_in, cnt_seg, q + 2, wn2);
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
                const uint32_t cntl = (uint32_t)__popcll(lanes);
                uint32_t base;
                bool ok;
                if (used + cntl <= pool_local) {
                    base = local0 + used;
                    used += cntl;
                    ok = true;
                } else {
                    // Overflow records of sample b live in their own slice, so
                    // the allocation atomics of different samples do not contend.
                    uint32_t ob = 0;
                    if (lane == 0) ob = atomicAdd(&pool_count[c.b], cntl);
                    ob = __shfl(ob, 0, kWave);
                    ok = (unsigned long long)ob + cntl <= (unsigned long long)pool_cap;
                    base = overflow0 + (uint32_t)c.b * pool_cap + ob;
                }
                if (lane == 0) {
                    WaveInfo wi;
                    wi.lanes = lanes;
                    wi.base = ok ? base : kNoSlot;
                    wi.pad = 0;
                    winfo[(((size_t)c.b * S + c.seg) * tiles + c.tile) * kSubPerSeg + q] = wi;
                }
                if (surv) {
                    // The entering state always; the full record if the pool
                    // had room (otherwise the resolve pass rebuilds the
                    // sub-block's states from the entering state).
                    ent[(((size_t)c.b * S + c.seg) * kSubPerSeg + q) * N + n] = make_double2(Vin, Iin);
                    if (ok) {
                        // Re-walk the sub-block to store its states.
                        uint32_t slot = base + (uint32_t)__popcll(lanes & below);
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
    if (n < N) mask[row + n] = msk;
    const bool want = ncand > 0 && n < N;
    if (__ballot(want)) {
        // Work list of sample b: the first segment to flag a neuron appends
        // it (one OR per flagged lane, then one counter update per wave).
        const size_t bn = (size_t)c.b * N + c.nc;
        const uint32_t old = atomicOr(&listed[bn], want ? 1u : 0u);
        const bool first = want && old == 0u;
        const unsigned long long fm = __ballot(first);
        if (fm) {
            uint32_t wbase = 0;
            if (lane == 0) wbase = atomicAdd(&nwork[c.b], (uint32_t)__popcll(fm));
            wbase = __shfl(wbase, 0, kWave);
            if (first) work[(size_t)c.b * N + wbase + (uint32_t)__popcll(fm & below)] = (uint32_t)bn;
        }
    }}

// ---------------------------------------------------------------------------
// Resolve pass: one wave per neuron that has flagged sub-blocks (a work list
// built by the check pass).  Intervals outside flagged sub-blocks provably
// hold no spike.  The flagged sub-blocks are taken in time order:
//   * Candidate list: the segments' sub-block masks are compacted into a
//     time-ordered list in LDS with one wave prefix sum per 64 segments.
//   * Chunks of kChunk candidates are processed one after the other, with
//     the loads of the next chunk in flight meanwhile.  Lane l holds
//     interval l % kSub of candidate 4 i + l / kSub of the chunk, i < 4 (the
//     four "slices"), so time order is (slice, lane).
//   * Each interval's maximum of h(u) = (V_lin(u) - th) e^{u/tm} is derived
//     in closed form once (interval_max); with D the deficit of the spikes
//     so far at the interval start, it crosses iff D a <= g.  A round takes
//     the earliest crossing interval (ballots), solves its spike time
//     (root_h) on its lane, emits the spike and raises that interval's own
//     deficit (so it is tested again for a second spike, Appendix E.2
//     restart); every later interval takes the new deficit with one
//     exponential.  Rounds repeat until no interval of the chunk crosses.
//   * The open interval after the last event is resolved last, on lane 0.
// Wave-uniform state: spike count, reset deficit dref right after the
// latest spike, at time tref.
// ---------------------------------------------------------------------------
constexpr int kCandCap = kWave * kSubPerSeg;     // candidates of 64 segments
constexpr int kSlices = 4;                       // intervals per lane in a chunk
constexpr int kChunk = kSlices * (kWave / kSub); // candidates per chunk

struct ResolveLds {
    uint32_t cand[kCandCap];                     // (segment in chunk << 3) | sub-block
};

// Rebuild a sub-block's entering no-reset state from its segment carry by
// walking the earlier events of the segment (used only when the record pool
// was full).
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

// Lane shift by n within rows of 16 lanes (DPP row_shr): lanes whose
// source lies outside the row keep `old`.
template <int n>
__device__ __forceinline__ double row_shr(double v, double old)
{
    static_assert(n >= 1 && n <= 15, "row shift");
    const unsigned long long u = (unsigned long long)__double_as_longlong(v);
    const unsigned long long o = (unsigned long long)__double_as_longlong(old);
    const int lo = __builtin_amdgcn_update_dpp((int)(unsigned)o, (int)(unsigned)u, 0x110 + n, 0xf, 0xf, false);
    const int hi = __builtin_amdgcn_update_dpp((int)(unsigned)(o >> 32), (int)(unsigned)(u >> 32), 0x110 + n, 0xf,
                                               0xf, false);
    return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}

// Affine map s -> (A V + C I + bV, D I + bI) of a run of events.
struct Map {
    double A, C, D, bV, bI;
};

// `late` applied after `early`.
__device__ __forceinline__ Map compose(const Map& late, const Map& early)
{
    Map r;
    r.A = late.A * early.A;
    r.C = late.A * early.C + late.C * early.D;
    r.D = late.D * early.D;
    r.bV = late.A * early.bV + late.C * early.bI + late.bV;
    r.bI = late.D * early.bI + late.bI;
    return r;
}

template <int n>
__device__ __forceinline__ Map row_shr_map(const Map& m)
{
    return Map{row_shr<n>(m.A, 1.0), row_shr<n>(m.C, 0.0), row_shr<n>(m.D, 1.0), row_shr<n>(m.bV, 0.0),
               row_shr<n>(m.bI, 0.0)};
}

// No-reset states of a sub-block whose record was not stored (pool full):
// lane j of each row of 16 lanes holds event j's map (Eq. affine: decay
// then jump), an inclusive scan over the row (Hillis-Steele with DPP row
// shifts; all 64 lanes take part) composes the maps of events 0..j, and the
// sub-block's entering state s0 gives the state after event j.  Lane j
// returns the state entering interval j (after event j - 1) and V at its end.
__device__ __forceinline__ double3 scan_interval(double2 s0, double A, double C, double D, double w)
{
    Map m{A, C, D, 0.0, w};
    m = compose(m, row_shr_map<1>(m));
    m = compose(m, row_shr_map<2>(m));
    m = compose(m, row_shr_map<4>(m));
    m = compose(m, row_shr_map<8>(m));
    const double Va = m.A * s0.x + m.C * s0.y + m.bV;     // after event j
    const double Ia = m.D * s0.y + m.bI;
    return make_double3(row_shr<1>(Va, s0.x), row_shr<1>(Ia, s0.y), Va);
}

__device__ __forceinline__ int rl_int(int v, int l) { return __builtin_amdgcn_readlane(v, l); }

__device__ __forceinline__ double rl_double(double v, int l)
{
    unsigned long long u = (unsigned long long)__double_as_longlong(v);
    unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)u, l);
    unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(u >> 32), l);
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// One lane's interval: start time and length, no-reset state at its start
// (V0, I0) and end (V1), decays of its gap.
struct Iv {
    double t0, L, V0, I0, V1, A, D;
    bool valid;
};

// The raw loads of one lane's interval.  Every load is unconditional (from
// a clamped, valid address) and nothing is derived from the loaded values
// until the interval is used: a branch around a load, or a select of its
// value, would make the compiler wait for every outstanding load at that
// point, which defeats the prefetch of the next chunk.
struct IvRaw {
    float tp, tb;       // time of the previous event and of this interval's event
    double A, D;        // decays of the gap
    double2 s0;         // record: no-reset state at the interval start
    double v1;          // record: no-reset V at the interval end
    int k, seg, kq0, cnt, j;
    bool valid, fb;     // fb: the record pool was full for this sub-block
    bool rowfb;         // the same for the lane's row, valid or not
};

// The window's per-candidate values (one candidate per lane).
struct WinLane {
    int kq0, cnt, seg;
    uint32_t slot;
};

__device__ __forceinline__ IvRaw load_slice(int cw, int nwin, const WinLane& w, int j, const float* __restrict__ tt,
                                            const Decay* __restrict__ d, const Record* __restrict__ pool)
{
    IvRaw v;
    const int c = min(cw, kWave - 1);
    v.kq0 = __shfl(w.kq0, c, kWave);
    v.cnt = __shfl(w.cnt, c, kWave);
    v.seg = __shfl(w.seg, c, kWave);
    const uint32_t slot = (uint32_t)__shfl((int)w.slot, c, kWave);
    v.j = j;
    v.valid = cw < nwin && j < v.cnt;
    v.fb = v.valid && slot == kNoSlot;
    v.rowfb = cw < nwin && slot == kNoSlot;
    v.k = v.kq0 + (v.valid ? j : 0);
    v.tp = tt[max(v.k - 1, 0)];
    v.tb = tt[v.k];
    v.A = d[v.k].A;
    v.D = d[v.k].D;
    const Record* rec = pool + (v.valid && slot != kNoSlot ? slot : 0u);   // pool holds at least one record
    v.s0 = rec->s[j];
    v.v1 = rec->s[j + 1].x;
    return v;
}

__device__ __forceinline__ Iv finish_slice(const IvRaw& r, int b, int n, int S, int N, int C_in,
                                           const int32_t* __restrict__ src, const Decay* __restrict__ d,
                                           const float* __restrict__ WT, const double2* __restrict__ ent)
{
    Iv v;
    v.valid = r.valid;
    v.t0 = r.k > 0 ? (double)r.tp : 0.0;
    v.L = (double)r.tb - v.t0;
    v.A = r.A;
    v.D = r.D;
    v.V0 = r.s0.x;
    v.I0 = r.s0.y;
    v.V1 = r.v1;
    if (__ballot(r.rowfb)) {
        // No record: rebuild the row's states from its entering state (every
        // lane takes part in the row scan; past cnt the maps are identities).
        const int q = (r.kq0 % kSeg) / kSub;
        const double2 s0 = r.rowfb ? ent[(((size_t)b * S + r.seg) * kSubPerSeg + q) * N + n] : make_double2(0.0, 0.0);
        const bool in = r.j < r.cnt;
        const int k = r.kq0 + min(r.j, max(r.cnt - 1, 0));
        const Decay e = d[k];
        const double w = in ? (double)WT[(size_t)clamp_src(src[k], C_in) * (size_t)N + n] : 0.0;
        const double3 sc = scan_interval(s0, in ? e.A : 1.0, in ? e.C : 0.0, in ? e.D : 1.0, w);
        if (r.fb) { v.V0 = sc.x; v.I0 = sc.y; v.V1 = sc.z; }
    }
    return v;
}

// Float32 screen of the interval test D a <= g, with no transcendental
// function.  The crossing condition is D <= max of h over the interval.
// h(L) = (V_lin(L) - th) e^{L/tm} is known exactly (the end test
// D e^{-L/tm} <= V_lin(L) - th); when I0 > th, h is concave with
// h'(0) = (I0 - th)/tm > 0, so its tangent at 0 bounds it over the whole
// interval: max h <= V0 - th + (I0 - th) L / tm.  An interval that misses
// both tests by more than 1e-4 of the magnitude of their terms (far above
// float32 rounding of these few operations and of the hardware exp used for
// D) cannot cross; only the others are tested exactly in float64.
struct Screen {
    float e_rhs, e_a, e_s;   // end test:     D e_a <= e_rhs  (+ margin on e_s)
    float i_rhs, i_s;        // tangent test: D <= i_rhs      (+ margin on i_s), when I0 > th
    bool tangent;
};

__device__ __forceinline__ Screen screen32(const Model& m, const Iv& v)
{
    const float V0 = (float)v.V0, I0 = (float)v.I0, V1 = (float)v.V1, L = (float)v.L;
    const float th = m.f_th, Lt = L * m.f_inv_tm;
    Screen c;
    c.e_rhs = V1 - th;
    c.e_a = (float)v.A;
    c.e_s = fabsf(V1) + th;
    c.tangent = I0 > th * (1.0f - 1e-5f);
    c.i_rhs = (V0 - th) + (I0 - th) * Lt;
    c.i_s = fabsf(V0) + th + fabsf(I0) * Lt;
    return c;
}

// Reset deficit at time t0 in float32 (0 before the first spike).
__device__ __forceinline__ float deficit32(int ns, double dref, double tref, double t0, const Model& m)
{
    return ns > 0 ? (float)dref * __expf((float)(-(t0 - tref) * m.inv_tm)) : 0.0f;
}

__device__ __forceinline__ bool may_cross(const Screen& c, float D)
{
    const float da = D * c.e_a;
    const bool end_miss = da - c.e_rhs > 1e-4f * (c.e_s + da);
    const bool tan_miss = !c.tangent || D - c.i_rhs > 1e-4f * (c.i_s + D);
    return !(end_miss && tan_miss);      // NaN passes (tested in float64)
}

// Status counts of one wave, added to the status words once per wave.
struct ResolveStats {
    int walked, fallback, capped, spikes;
};

__device__ void resolve_neuron(ResolveLds& sh, ResolveStats& acc, int b, int n, const float* __restrict__ ev_t,
                               const int32_t* __restrict__ ev_src, const int32_t* __restrict__ ev_n, int E_max,
                               const float* __restrict__ WT, int C_in, int N, int tiles, int S, const Model& m,
                               const Decay* __restrict__ dec, const double2* __restrict__ carry,
                               const double2* __restrict__ ent,
                               const uint32_t* __restrict__ mask, const WaveInfo* __restrict__ winfo,
                               const Record* __restrict__ pool, float* __restrict__ out_t, int32_t* __restrict__ out_n,
                               float* __restrict__ out_i)
{
    const int tile = n / kWave;
    const unsigned long long below_n = (1ull << (n % kWave)) - 1ull;
    const int lane = (int)threadIdx.x;
    const int j = lane % kSub, r = lane / kSub;
    const int nb = clamp_count(ev_n[b], E_max);
    const float* tt = ev_t + (size_t)b * E_max;
    const int32_t* src = ev_src + (size_t)b * E_max;
    const Decay* d = dec + (size_t)b * E_max;
    const size_t idx = (size_t)b * N + n;
    float* st = out_t + idx * (size_t)m.s_max;
    float* si = out_i ? out_i + idx * (size_t)m.s_max : nullptr;
    const int Sb = (nb + kSeg - 1) / kSeg;

    int ns = 0, walked = 0, fallback = 0;
    bool capped = false, last_seen = false;
    int last_seg = 0, last_cnt = 0;
    uint32_t last_slot = kNoSlot;
    double dref = 0.0, tref = 0.0;     // deficit right after the latest spike, its time

    for (int seg0 = 0; seg0 < Sb && !capped; seg0 += kWave) {
        // ---- compact this chunk's flagged sub-blocks into a time-ordered list
        const int sj = seg0 + lane;
        const uint32_t mv = sj < Sb ? mask[((size_t)b * S + sj) * N + n] : 0u;
        const int pc = __popc(mv);
        int ex = pc;
#pragma unroll
        for (int off = 1; off < kWave; off <<= 1) {
            int v = __shfl_up(ex, off, kWave);
            if (lane >= off) ex += v;
        }
        const int tot = rl_int(ex, kWave - 1);
        ex -= pc;
        {
            uint32_t mm = mv;
            int o = ex;
            while (mm) {
                sh.cand[o++] = ((uint32_t)lane << 3) | (uint32_t)__builtin_ctz(mm);
                mm &= mm - 1u;
            }
        }
        __syncthreads();

        for (int w0 = 0; w0 < tot && !capped; w0 += kWave) {
            // ---- window: lane c holds candidate w0 + c
            const int nwin = min(kWave, tot - w0);
            WinLane w{0, 0, 0, kNoSlot};
            bool last = false;
            if (lane < nwin) {
                uint32_t cw = sh.cand[w0 + lane];
                w.seg = seg0 + (int)(cw >> 3);
                int q = (int)(cw & 7u);
                w.kq0 = w.seg * kSeg + q * kSub;
                w.cnt = min(kSub, nb - w.kq0);
                WaveInfo wi = winfo[(((size_t)b * S + w.seg) * tiles + tile) * kSubPerSeg + q];
                if (wi.base != kNoSlot) w.slot = wi.base + (uint32_t)__popcll(wi.lanes & below_n);
                last = w.kq0 + w.cnt == nb;
            }
            fallback += __popcll(__ballot(lane < nwin && w.slot == kNoSlot));
            {
                unsigned long long lm = __ballot(last);
                if (lm) {
                    const int ll = __ffsll((long long)lm) - 1;
                    last_seen = true;
                    last_seg = rl_int(w.seg, ll);
                    last_cnt = rl_int(w.cnt, ll);
                    last_slot = (uint32_t)rl_int((int)w.slot, ll);
                }
            }

            IvRaw nx[kSlices];
#pragma unroll
            for (int i = 0; i < kSlices; ++i) nx[i] = load_slice(i * (kWave / kSub) + r, nwin, w, j, tt, d, pool);
            for (int c0 = 0; c0 < nwin && !capped; c0 += kChunk) {
                IvRaw raw[kSlices];
#pragma unroll
                for (int i = 0; i < kSlices; ++i) raw[i] = nx[i];
                walked += min(kChunk, nwin - c0);
                // ---- prefetch the next chunk
                if (c0 + kChunk < nwin) {
#pragma unroll
                    for (int i = 0; i < kSlices; ++i)
                        nx[i] = load_slice(c0 + kChunk + i * (kWave / kSub) + r, nwin, w, j, tt, d, pool);
                }
                Iv v[kSlices];
#pragma unroll
                for (int i = 0; i < kSlices; ++i) v[i] = finish_slice(raw[i], b, n, S, N, C_in, src, d, WT, ent);
                // ---- slices in time order: screen in float32 with the current
                // deficit, then the deficit and the maximum in float64 where
                // an interval may cross, then rounds
#pragma unroll
                for (int i = 0; i < kSlices; ++i) {
                    if (capped) break;
                    const Iv& x = v[i];
                    const Screen sc = screen32(m, x);
                    bool pend = x.valid && x.L > 0.0 && may_cross(sc, deficit32(ns, dref, tref, x.t0, m));
                    if (!__ballot(pend)) continue;
                    double Dl = 0.0, lo = 0.0, Flo = 0.0;
                    IntervalMax im{-1.0, 1.0, 0.0, 0.0};
                    if (pend) {
                        Dl = ns > 0 ? dref * exp(-(x.t0 - tref) * m.inv_tm) : 0.0;
                        im = interval_max(m, x.V0, x.I0, x.V1, x.L, x.A, x.D);
                        Flo = x.V0 - m.th - Dl;
                    }
                    // ---- rounds: the earliest crossing lane solves, the later
                    // ones re-test
                    for (;;) {
                        const unsigned long long cm = __ballot(pend && Dl * im.a <= im.g);
                        if (!cm) break;
                        const int kl = __ffsll((long long)cm) - 1;
                        double tsp = 0.0, dnew = 0.0;
                        if (lane == kl) {
                            double E1, E2;
                            const double kI = m.kappa * x.I0;
                            const double u = root_h(m, x.V0 - Dl + kI, kI, lo, Flo, im.hi, im.Fhi - Dl, &E1, &E2,
                                                    nullptr);
                            const double iE1 = rcp_refined(E1);
                            tsp = x.t0 + u;
                            st[ns] = (float)tsp;
                            if (si) si[ns] = (float)(x.I0 * (E2 * iE1));
                            dnew = Dl * iE1 + m.dth;
                            // the same interval is tested again with the raised deficit
                            Dl += m.dth * E1;
                            lo = u;
                            Flo = -m.dth * E1;
                        }
                        ++ns;
                        dref = rl_double(dnew, kl);
                        tref = rl_double(tsp, kl);
                        if (ns >= m.s_max) { capped = true; break; }
                        if (lane < kl) pend = false;
                        if (pend && lane > kl) {
                            pend = may_cross(sc, deficit32(ns, dref, tref, x.t0, m));
                            if (__ballot(pend) && pend) {
                                Dl = dref * exp(-(x.t0 - tref) * m.inv_tm);
                                Flo = x.V0 - m.th - Dl;
                            }
                        }
                    }
                }
            }
        }
        __syncthreads();                              // the list is rewritten by the next chunk
    }

    // ---- the open interval (t_last, t_end] after the last event, lane 0
    const double t_last = nb > 0 ? (double)tt[nb - 1] : 0.0;
    if (!capped && last_seen && m.t_end > t_last && lane == 0) {
        double2 s0 = last_slot != kNoSlot
                         ? pool[last_slot].s[last_cnt]
                         : entering_state(carry, ((size_t)b * S + last_seg) * N, n, last_seg * kSeg, nb, src, d, WT,
                                          C_in, N);
        const double V0 = s0.x, I0 = s0.y, L = m.t_end - t_last;
        double A = 0.0, Dd = 0.0, V1 = 0.0;
        if (!isinf(L)) {
            A = exp(-L * m.inv_tm);
            Dd = exp(-L * m.inv_ts);
            V1 = V0 * A + unit_kernel(m, L, A) * I0;
        }
        const IntervalMax im = interval_max(m, V0, I0, V1, L, A, Dd);
        double Dk = ns > 0 ? dref * exp(-(t_last - tref) * m.inv_tm) : 0.0;
        double lo = 0.0, Flo = V0 - m.th - Dk;
        const double kI = m.kappa * I0;
        while (Dk * im.a <= im.g) {
            double E1, E2;
            double u = root_h(m, V0 - Dk + kI, kI, lo, Flo, im.hi, im.Fhi - Dk, &E1, &E2, nullptr);
            st[ns] = (float)(t_last + u);
            if (si) si[ns] = (float)(I0 * (E2 * rcp_refined(E1)));
            ++ns;
            Dk += m.dth * E1;
            lo = u;
            Flo = -m.dth * E1;
            if (ns >= m.s_max) { capped = true; break; }
        }
    }
    ns = rl_int(ns, 0);
    capped = rl_int((int)capped, 0) != 0;

    if (lane == 0) out_n[idx] = ns;
    acc.walked += walked;
    acc.fallback += fallback;
    acc.capped += capped ? 1 : 0;
    acc.spikes += ns;
}

// Work-list driven: the per-sample lists of neurons built by k_check are
// taken as one concatenated list, entry w by workgroup w mod gridDim.x, so
// that samples with many listed neurons spread over the whole grid.  Status
// counts are added once per workgroup.
__global__ __launch_bounds__(kWave) void k_resolve(const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src,
                                                   const int32_t* __restrict__ ev_n, int B, int E_max,
                                                   const float* __restrict__ WT, int C_in, int N, int tiles, int S,
                                                   Model m, const Decay* __restrict__ dec,
                                                   const double2* __restrict__ carry,
                                                   const double2* __restrict__ ent,
                                                   const uint32_t* __restrict__ mask,
                                                   const WaveInfo* __restrict__ winfo,
                                                   const Record* __restrict__ pool,
                                                   const uint32_t* __restrict__ work, const uint32_t* __restrict__ nwork,
                                                   float* __restrict__ out_t, int32_t* __restrict__ out_n,
                                                   float* __restrict__ out_i, int32_t* __restrict__ status)
{
    __shared__ ResolveLds sh;
    const int lane = (int)threadIdx.x;
    ResolveStats acc{0, 0, 0, 0};
    // Running sum of the list lengths over groups of 64 samples (one load
    // per lane, a wave prefix sum): entry w of the concatenated lists belongs
    // to the first sample whose running sum exceeds w.
    int b0 = 0;               // first sample of the current group
    uint32_t base = 0;        // entries of the samples before the group
    uint32_t incl = 0;        // running sum up to and including sample b0 + lane
    auto load_group = [&]() {
        uint32_t c = b0 + lane < B ? nwork[b0 + lane] : 0u;
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
        const uint32_t bn = work[(size_t)b * N + (w - before)];
        resolve_neuron(sh, acc, (int)(bn / (uint32_t)N), (int)(bn % (uint32_t)N), ev_t, ev_src, ev_n, E_max, WT,
                       C_in, N, tiles, S, m, dec, carry, ent, mask, winfo, pool, out_t, out_n, out_i);
    }
    if (threadIdx.x == 0) {
        if (acc.walked) {
            atomicAdd(&status[LIF_ST_WALKED_BLOCKS], acc.walked);
            atomicAdd(&status[LIF_ST_CAND_BLOCKS], acc.walked);
        }
        if (acc.fallback) atomicAdd(&status[LIF_ST_POOL_FALLBACK], acc.fallback);
        if (acc.capped) {
            atomicAdd(&status[LIF_ST_CAPPED], acc.capped);
            atomicOr(&status[LIF_ST_FLAGS], LIF_WARN_SPIKE_CAP);
        }
        if (acc.spikes) {
            atomicAdd(&status[LIF_ST_SPIKES], acc.spikes);
            atomicAdd(&status[LIF_ST_ROOT_SOLVES], acc.spikes);
        }
    }
}

// Sequential baseline (Appendix E.3): one thread per (sample, neuron)
// consumes every event in order with the same interval test and root solve.
// The state (V, I) is the true one, so each interval starts with deficit 0;
// spikes inside it raise the deficit and the rest of the interval is
// re-tested.
__global__ __launch_bounds__(64) void k_sequential(const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src,
                                                   const int32_t* __restrict__ ev_n, int B, int E_max,
                                                   const float* __restrict__ WT, int C_in, int N, Model m,
                                                   const Decay* __restrict__ dec, float* __restrict__ out_t,
                                                   int32_t* __restrict__ out_n, float* __restrict__ out_i,
                                                   int32_t* __restrict__ status)
{
    const size_t idx_raw = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const bool live = idx_raw < (size_t)B * (size_t)N;
    const size_t idx = live ? idx_raw : 0;            // lanes past the end run neuron 0 and write nothing
    int b = (int)(idx / (size_t)N), n = (int)(idx % (size_t)N);
    int nb = clamp_count(ev_n[b], E_max);
    if (live && n == 0) atomicAdd(&status[LIF_ST_EVENTS], nb);
    const float* tt = ev_t + (size_t)b * E_max;
    const int32_t* src = ev_src + (size_t)b * E_max;
    const Decay* d = dec + (size_t)b * E_max;
    float* st = out_t + idx * (size_t)m.s_max;
    float* si = out_i ? out_i + idx * (size_t)m.s_max : nullptr;
    int ns = 0;
    bool capped = false;
    double V = 0.0, I = 0.0, t_prev = 0.0;
    for (int k = 0; k <= nb && !capped; ++k) {
        double L, A, C, Dd, gb;
        if (k < nb) {
            Decay e = d[k];
            A = e.A; C = e.C; Dd = e.D; gb = e.g;
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
            double gl = fmin(L, m.t_peak);
            gb = unit_kernel(m, gl, exp(-gl * m.inv_tm)) * (1.0 + 1e-12);
        }
        double V1 = A * V + C * I;
        if (L > 0.0 && fmax(V, 0.0) + fmax(I, 0.0) * gb >= m.th_lo) {
            IntervalMax im = interval_max(m, V, I, V1, L, A, Dd);
            double Dk = 0.0, lo = 0.0, Flo = V - m.th;
            const double kI = m.kappa * I;
            while (Dk * im.a <= im.g) {
                double E1, E2;
                double u = root_h(m, V - Dk + kI, kI, lo, Flo, im.hi, im.Fhi - Dk, &E1, &E2, nullptr);
                if (live) {
                    st[ns] = (float)(t_prev + u);
                    if (si) si[ns] = (float)(I * (E2 / E1));
                }
                ++ns;
                Dk += m.dth * E1;
                lo = u;
                Flo = -m.dth * E1;
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
        }
    }
    // status counts: one atomic per wave
    int nsw = live ? ns : 0, cw = live && capped ? 1 : 0;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        nsw += __shfl_xor(nsw, off, kWave);
        cw += __shfl_xor(cw, off, kWave);
    }
    if (threadIdx.x % kWave == 0) {
        if (cw) {
            atomicAdd(&status[LIF_ST_CAPPED], cw);
            atomicOr(&status[LIF_ST_FLAGS], LIF_WARN_SPIKE_CAP);
        }
        if (nsw) {
            atomicAdd(&status[LIF_ST_SPIKES], nsw);
            atomicAdd(&status[LIF_ST_ROOT_SOLVES], nsw);
        }
    }
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
    L.ent = take((size_t)B * L.S * kSubPerSeg * N * sizeof(double2));
    int tiles = (N + kWave - 1) / kWave;
    L.winfo = take((size_t)B * L.S * tiles * kSubPerSeg * sizeof(WaveInfo));
    L.counters = take(2 * (size_t)B * sizeof(uint32_t));   // per sample: pool use, work-list length
    L.listed = take((size_t)B * N * sizeof(uint32_t));
    L.work = take((size_t)B * N * sizeof(uint32_t));
    // Record pool: one record per flagged (sub-block, neuron).  Each check
    // wave (sample, segment, tile) owns kPoolLocal slots; the overflow is
    // shared per sample and sized at a 64th of the dense bound (far above
    // what spiking activity needs).  A full pool only sends the excess
    // sub-blocks through a slower re-walk.  LIF_POOL_LOCAL / LIF_POOL_CAP
    // override the two sizes (used by tests of the re-walk path).
    size_t local = kPoolLocal;
    if (const char* env = getenv("LIF_POOL_LOCAL")) local = (size_t)strtoull(env, nullptr, 10);
    size_t waves = (size_t)B * L.S * tiles;
    size_t dense = waves * kSubPerSeg * kWave;
    size_t cap = dense / 64 > 65536 ? dense / 64 : (dense < 65536 ? dense : 65536);
    if (const char* env = getenv("LIF_POOL_CAP")) cap = (size_t)strtoull(env, nullptr, 10);
    if (local > 64) local = 64;
    if (waves * local + cap > 0xfffffff0ull) cap = 0xfffffff0ull - waves * local;   // slot indices are 32-bit
    L.pool_local = local;
    L.pool_cap = cap;
    size_t recs = waves * local + cap;
    L.pool = take((recs > 0 ? recs : 1) * sizeof(Record));   // at least one record (a safe load address)
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
    double2* ent = (double2*)(base + L.ent);
    uint32_t* mask = (uint32_t*)(base + L.mask);
    WaveInfo* winfo = (WaveInfo*)(base + L.winfo);
    uint32_t* counters = (uint32_t*)(base + L.counters);
    uint32_t* pool_count = counters;
    uint32_t* nwork = counters + B;
    uint32_t* listed = (uint32_t*)(base + L.listed);
    uint32_t* work = (uint32_t*)(base + L.work);
    Record* pool = (Record*)(base + L.pool);

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
        TIMED_LAUNCH("carry", k_carry, dim3((unsigned)((size_t)B * tiles)), dim3(kWave * kCarryWaves), 0, stream,
                     ev_n, B, E_max, N, tiles, L.S, segm, agg, carry, status, out_n, listed, counters);
    if (total) {
        TIMED_LAUNCH("check", k_check, dim3((unsigned)total), dim3(kWave * kTilesPerBlock), 0, stream,
                     ev_t, ev_src, ev_n, E_max, WT, C_in, N, tiles, tgroups, L.S, (int)total, m, dec, carry, ent, mask,
                     winfo, pool, pool_count, (uint32_t)L.pool_local, (uint32_t)(L.pool_cap / (B > 0 ? B : 1)),
                     listed, work, nwork,
                     status);
        // Single-wave workgroups over the concatenated per-sample lists.
        const unsigned rgrid = (unsigned)(nn < 4096 ? nn : 4096);
        TIMED_LAUNCH("resolve", k_resolve, dim3(rgrid), dim3(kWave), 0, stream,
                     ev_t, ev_src, ev_n, B, E_max, WT, C_in, N, tiles, L.S, m, dec, carry, ent, mask, winfo, pool,
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
