// lif_delay.hip -- a layer with learnable synaptic delays (Sec. 3.1 Eq.
// spike_input: a spike of input channel j at t_k reaches neuron i at
// t_k + d_ij; Appendix E.2: a sorted event queue per neuron; Appendix E.5:
// delays per layer, initialised uniformly in [0, 0.1] s).
//
// Delays break what the main forward is built on: the event maps are no
// longer shared by the neurons of a sample, since every neuron sees its own
// event order.  The delayed layer therefore runs per neuron:
//   k_dly_arrival  per (sample, 64 events, 64 neurons): the arrivals
//                  a = fl32(t_k + d_ij), with the delays read as coalesced
//                  W^T-layout row slices (lanes = neurons) and written per
//                  neuron through an LDS transpose (lanes = events), so both
//                  sides are coalesced.
//   k_dly_queue_lds / k_dly_queue
//                  per (sample, neuron), one workgroup: the neuron's queue,
//                  its events ordered by the key (arrival bits, then k), by a
//                  bucket sort: arrivals are binned by value (a histogram and
//                  a prefix sum in LDS), scattered into their bins, and each
//                  key is then placed at its bin's start plus its rank among
//                  the bin's keys.  Keys are unique, so the result does not
//                  depend on the order in which the scatter's atomics land.
//                  Queues of up to kQLdsMax events keep their keys in
//                  registers and the binned keys in LDS (one read of the
//                  arrivals); longer ones bin through global memory.
//   forward        the chunked walk of lif_chunked.hip on these queues (one
//                  wave per neuron, K = 128 events per iteration, no budget:
//                  every event is consumed unless the neuron stops at s_max).
//   k_dly_adjoint  per (sample, neuron) that fires: the adjoint sums
//                  P^m_r = sum over the spikes s after queue event r of
//                  mu_s e^{-(t_s - a_r)/tm} (P^s_r the same with ts), taken
//                  64 queue events per step from the last one that feeds a
//                  spike down to the first (lanes = events), from a carry of
//                  the later spikes plus the spikes that fall inside the step;
//                  for queue event r with channel j and sample index k:
//                    dL/dw_ij += kappa (P^m_r - P^s_r)
//                    dL/dd_ij += w_ij kappa (P^m_r / tm - P^s_r / ts)  (= dL/da_r)
//                    dL/dt_k  += the same dL/da_r
//                  added as 64-bit fixed-point integers (exact and order
//                  free, so the gradients are bitwise reproducible) with
//                  power-of-two scales that keep every sum below 2^62.
#include "lif_common.hpp"
#include "lif_host.hpp"
#include "lif_reg.hpp"
#include "lif_scan.hpp"

namespace lif {

constexpr int kQThreads = 256;
constexpr int kQBins = 8192;            // most bins of one queue's bucket sort (32 KB of LDS)

// Arrival of event k at neuron n: the float32 sum (no contraction is
// possible in a single add); -0 becomes +0 so that the bits order like the
// values for every non-negative arrival.
__device__ __forceinline__ float arrival(const float* __restrict__ tt, const int32_t* __restrict__ src,
                                         const float* __restrict__ DT, int C_in, int N, int n, int k)
{
    const float a = tt[k] + DT[(size_t)clamp_src(src[k], C_in) * (size_t)N + n];
    return a + 0.0f;
}

// Bin of an arrival: floor(a * sc) clamped into [0, nbins - 1]; monotone
// non-decreasing in a (a NaN or negative value goes to bin 0).
__device__ __forceinline__ int bin_of(float a, float sc, int nbins)
{
    const float x = a * sc;
    if (!(x >= 0.0f)) return 0;
    return x < (float)(nbins - 1) ? (int)x : nbins - 1;
}

constexpr int kArrTile = 64;            // events and neurons per k_dly_arrival workgroup

__global__ __launch_bounds__(256) void k_dly_arrival(const float* __restrict__ ev_t,
                                                    const int32_t* __restrict__ ev_src,
                                                    const int32_t* __restrict__ ev_n, int E_max,
                                                    const float* __restrict__ DT, int C_in, int N,
                                                    float* __restrict__ arr)
{
    __shared__ float s_a[kArrTile][kArrTile + 1];      // [neuron][event]
    const int lane = (int)threadIdx.x % kWave, wave = (int)threadIdx.x / kWave;
    const int k0 = blockIdx.x * kArrTile, b = blockIdx.y, n0 = blockIdx.z * kArrTile;
    const int nb = clamp_count(ev_n[b], E_max);
    if (k0 >= nb) return;
    const float* tt = ev_t + (size_t)b * E_max;
    const int32_t* src = ev_src + (size_t)b * E_max;
    const int n = n0 + lane;
    for (int e = wave; e < kArrTile; e += 256 / kWave) {
        const int k = k0 + e;
        if (k < nb && n < N) s_a[lane][e] = arrival(tt, src, DT, C_in, N, n, k);
    }
    __syncthreads();
    const int k = k0 + lane;
    for (int q = wave; q < kArrTile; q += 256 / kWave) {
        const int nn = n0 + q;
        if (k < nb && nn < N) arr[((size_t)b * N + nn) * (size_t)E_max + k] = s_a[q][lane];
    }
}

// Queues of up to kMax events are sorted in registers and LDS by kThreads
// threads (kMax / kThreads arrivals each, kBins bins at most): 8192 by 512
// threads and 11520 by 768 (two workgroups per CU), 16384 by 1024 (112 KB of
// LDS, one).  Each sort is launched over every (sample, neuron) for which E_max
// allows a queue in its range and takes those whose queue length (the
// sample's event count) is above kMin and at most kMax, so that short queues
// get the sort with the most workgroups per CU whatever E_max is.
constexpr int kQLdsMax = 16384;         // longest queue sorted in registers and LDS

template <int kMin, int kMax, int kThreads, int kBins, int kWavesPerEU>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(kWavesPerEU))) void k_dly_queue_lds(const int32_t* __restrict__ ev_n, int E_max, int N,
                                                               const float* __restrict__ arr,
                                                               float* __restrict__ q_t, int32_t* __restrict__ q_k)
{
    constexpr int kQLdsBins = kBins;
    constexpr int kQR = kMax / kThreads;
    static_assert(kQR * kThreads == kMax && (kBins & (kBins - 1)) == 0 && kMax < 32768, "queue sort shape");
    __shared__ uint32_t s_at[kMax];        // binned arrivals (bits)
    __shared__ uint16_t s_ak[kMax];        // and their event indices
    __shared__ int s_bin[kQLdsBins];
    __shared__ float s_red[kThreads / kWave];
    __shared__ int s_wsum[kThreads / kWave];
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    const size_t item = blockIdx.x;
    const int b = (int)(item / (size_t)N);
    const int nb = clamp_count(ev_n[b], E_max);
    if (nb <= kMin || nb > kMax) return;      // empty, or another sort's range
    const size_t base = item * (size_t)E_max;
    // the thread's arrivals (event k = tid + r kThreads), all loads at once
    uint32_t ab[kQR];
#pragma unroll
    for (int r = 0; r < kQR; ++r) {
        const int k = tid + r * kThreads;
        ab[r] = k < nb ? __float_as_uint(arr[base + k]) : 0u;
    }
    float mx = 0.0f;
#pragma unroll
    for (int r = 0; r < kQR; ++r) mx = fmaxf(mx, __uint_as_float(ab[r]));
    for (int off = kWave / 2; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, kWave));
    if (lane == 0) s_red[wave] = mx;
    int nbins = 1;
    while (nbins < nb && nbins < kQLdsBins) nbins <<= 1;
    for (int j = tid; j < nbins; j += kThreads) s_bin[j] = 0;
    __syncthreads();
    float amax = s_red[0];
    for (int w = 1; w < kThreads / kWave; ++w) amax = fmaxf(amax, s_red[w]);
    const float sc = amax > 0.0f && amax < INFINITY ? (float)nbins / amax : 0.0f;
    int bin[kQR];
#pragma unroll
    for (int r = 0; r < kQR; ++r) {
        bin[r] = bin_of(__uint_as_float(ab[r]), sc, nbins);
        if (tid + r * kThreads < nb) atomicAdd(&s_bin[bin[r]], 1);
    }
    __syncthreads();
    // exclusive prefix sum over the bins: each thread a contiguous range,
    // the ranges' sums scanned across each wave, then over the waves
    const int per = (nbins + kThreads - 1) / kThreads;
    const int j0 = min(tid * per, nbins), j1 = min(j0 + per, nbins);
    int local = 0;
    for (int j = j0; j < j1; ++j) local += s_bin[j];
    int incl = local;
    for (int off = 1; off < kWave; off <<= 1) {
        const int x = __shfl_up(incl, off, kWave);
        if (lane >= off) incl += x;
    }
    if (lane == kWave - 1) s_wsum[wave] = incl;
    __syncthreads();
    int run = incl - local;
    for (int w = 0; w < wave; ++w) run += s_wsum[w];
    for (int j = j0; j < j1; ++j) {
        const int c = s_bin[j];
        s_bin[j] = run;
        run += c;
    }
    __syncthreads();
    // scatter into the bins in LDS; s_bin[j] ends at the end of bin j
#pragma unroll
    for (int r = 0; r < kQR; ++r) {
        const int k = tid + r * kThreads;
        if (k < nb) {
            const int pos = atomicAdd(&s_bin[bin[r]], 1);
            if (pos < nb) {
                s_at[pos] = ab[r];
                s_ak[pos] = (uint16_t)k;
            }
        }
    }
    __syncthreads();
    // each event's place: its bin's start plus its rank among the bin's
    // keys, the thread's events stepping through their bins together
    // (a bin's start and size packed as start | size << 16: both <= kMax < 2^15)
    int lc[kQR], rank[kQR];
    int mxc = 0;
#pragma unroll
    for (int r = 0; r < kQR; ++r) {
        const bool v = tid + r * kThreads < nb;
        const int lo = bin[r] > 0 ? s_bin[bin[r] - 1] : 0;
        const int cnt = v ? s_bin[bin[r]] - lo : 0;
        lc[r] = lo | (cnt << 16);
        rank[r] = 0;
        mxc = max(mxc, cnt);
    }
    for (int q = 0; q < mxc; ++q) {
#pragma unroll
        for (int r = 0; r < kQR; ++r) {
            if (q < (lc[r] >> 16)) {
                const int at = (lc[r] & 0xffff) + q;
                const uint32_t o = s_at[at];
                const int ok = s_ak[at];
                rank[r] += o < ab[r] || (o == ab[r] && ok < tid + r * kThreads);
            }
        }
    }
    __syncthreads();
    // the queue in order in LDS, then written out coalesced
#pragma unroll
    for (int r = 0; r < kQR; ++r) {
        const int place = (lc[r] & 0xffff) + rank[r];
        if ((lc[r] >> 16) > 0 && place < nb) {  // always: a key's bin is the one it was scattered to
            s_at[place] = ab[r];
            s_ak[place] = (uint16_t)(tid + r * kThreads);
        }
    }
    __syncthreads();
    for (int i = tid; i < nb; i += kThreads) {
        q_t[base + i] = __uint_as_float(s_at[i]);
        q_k[base + i] = s_ak[i];
    }
}

// 64-bit sort key of event k with arrival a: the arrival's bits (which order
// like the values for non-negative arrivals), then k.
__device__ __forceinline__ unsigned long long arrival_key(float a, int k)
{
    return ((unsigned long long)__float_as_uint(a) << 32) | (unsigned)k;
}

__global__ __launch_bounds__(kQThreads) void k_dly_queue(const int32_t* __restrict__ ev_n, int E_max, int N,
                                                        const float* __restrict__ arr,
                                                        unsigned long long* __restrict__ keys,
                                                        float* __restrict__ q_t, int32_t* __restrict__ q_k)
{
    __shared__ int s_bin[kQBins];
    __shared__ float s_red[kQThreads / kWave];
    __shared__ int s_part[kQThreads];
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    const size_t item = blockIdx.x;
    const int b = (int)(item / (size_t)N);
    const int nb = clamp_count(ev_n[b], E_max);
    if (nb <= kQLdsMax) return;               // sorted in LDS
    const size_t base = item * (size_t)E_max;
    const float* ain = arr + base;
    auto key_arrival = [](unsigned long long key) { return __uint_as_float((unsigned)(key >> 32)); };
    // the largest arrival
    float mx = 0.0f;
    for (int k = tid; k < nb; k += kQThreads) mx = fmaxf(mx, ain[k]);
    for (int off = kWave / 2; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, kWave));
    if (lane == 0) s_red[wave] = mx;
    int nbins = 1;
    while (nbins < nb && nbins < kQBins) nbins <<= 1;
    for (int j = tid; j < nbins; j += kQThreads) s_bin[j] = 0;
    __syncthreads();
    float amax = s_red[0];
    for (int w = 1; w < kQThreads / kWave; ++w) amax = fmaxf(amax, s_red[w]);
    const float sc = amax > 0.0f && amax < INFINITY ? (float)nbins / amax : 0.0f;
    // histogram
    for (int k = tid; k < nb; k += kQThreads) atomicAdd(&s_bin[bin_of(ain[k], sc, nbins)], 1);
    __syncthreads();
    // exclusive prefix sum over the bins: each thread a contiguous range
    const int per = (nbins + kQThreads - 1) / kQThreads;
    const int j0 = min(tid * per, nbins), j1 = min(j0 + per, nbins);
    int local = 0;
    for (int j = j0; j < j1; ++j) local += s_bin[j];
    s_part[tid] = local;
    __syncthreads();
    for (int off = 1; off < kQThreads; off <<= 1) {
        const int x = tid >= off ? s_part[tid - off] : 0;
        __syncthreads();
        s_part[tid] += x;
        __syncthreads();
    }
    int run = s_part[tid] - local;
    for (int j = j0; j < j1; ++j) {
        const int c = s_bin[j];
        s_bin[j] = run;
        run += c;
    }
    __syncthreads();
    // scatter into the bins; s_bin[j] ends at the end of bin j
    for (int k = tid; k < nb; k += kQThreads) {
        const float a = ain[k];
        const int pos = atomicAdd(&s_bin[bin_of(a, sc, nbins)], 1);
        if (pos < nb) keys[base + pos] = arrival_key(a, k);
    }
    __syncthreads();
    // each key's place: its bin's start plus its rank among the bin's keys
    for (int p = tid; p < nb; p += kQThreads) {
        const unsigned long long key = keys[base + p];
        const int j = bin_of(key_arrival(key), sc, nbins);
        const int lo = j > 0 ? s_bin[j - 1] : 0, hi = s_bin[j];
        int rank = 0;
        for (int q = lo; q < hi; ++q) rank += keys[base + q] < key;
        if (lo + rank < nb) {                 // always: a key's bin is the one it was scattered to
            q_t[base + lo + rank] = key_arrival(key);
            q_k[base + lo + rank] = (int32_t)(key & 0xffffffffull);
        }
    }
}

// Status words of the queue build: events of the batch, and
// LIF_WARN_BAD_DELAY when a delay is negative or not finite.
__global__ __launch_bounds__(256) void k_dly_check(const float* __restrict__ DT, size_t nD,
                                                  const int32_t* __restrict__ ev_n, int B, int E_max,
                                                  int32_t* __restrict__ status)
{
    const size_t gtid = (size_t)blockIdx.x * blockDim.x + threadIdx.x, gs = (size_t)gridDim.x * blockDim.x;
    bool bad = false;
    for (size_t x = gtid; x < nD; x += gs) bad |= !(DT[x] >= 0.0f && DT[x] < INFINITY);
    if (__ballot(bad) && threadIdx.x % kWave == 0) atomicOr(&status[LIF_ST_FLAGS], LIF_WARN_BAD_DELAY);
    if (gtid == 0) {
        int ev = 0;
        for (int b = 0; b < B; ++b) ev += clamp_count(ev_n[b], E_max);
        atomicAdd(&status[LIF_ST_EVENTS], ev);
    }
}

__global__ void k_dly_status_reset(int32_t* __restrict__ status)
{
    if (threadIdx.x < LIF_STATUS_WORDS) status[threadIdx.x] = 0;
}

// ---------------------------------------------------------------------------
// Backward
// ---------------------------------------------------------------------------
struct DlyBwdLayout {
    size_t mu, musum, scale, wmax, gw, gd, gt, tcnt, tq, total;
};

// tq (the walks' per-queue-event dL/dt terms) comes last and only with
// want_t, so that a call without dL/dt can take B N E_max 8 bytes less.
static DlyBwdLayout dly_bwd_layout(int B, int E_max, int C_in, int N, int s_max, bool want_t)
{
    DlyBwdLayout L{};
    size_t off = 0;
    auto take = [&](size_t bytes) { size_t o = off; off += (bytes + 255) & ~(size_t)255; return o; };
    L.mu = take((size_t)B * N * s_max * sizeof(double));
    L.musum = take((size_t)B * N * sizeof(double));
    L.scale = take(4 * sizeof(double));
    L.wmax = take(sizeof(uint32_t));
    L.gw = take((size_t)C_in * N * sizeof(long long));
    L.gd = take((size_t)C_in * N * sizeof(long long));
    L.gt = take((size_t)B * E_max * sizeof(long long));
    L.tcnt = take((size_t)B * N * sizeof(int32_t));
    L.tq = take(want_t ? (size_t)B * N * (size_t)E_max * sizeof(long long) : 0);
    L.total = off + 256;
    return L;
}

// Zeroed accumulators and the spike adjoints of every (sample, neuron).
__global__ __launch_bounds__(256) void k_dly_setup(size_t nW, size_t nT, long long* __restrict__ gw,
                                                  long long* __restrict__ gd, long long* __restrict__ gt,
                                                  uint32_t* __restrict__ wmax, size_t nn, Model m,
                                                  const float* __restrict__ out_t, const int32_t* __restrict__ out_n,
                                                  const float* __restrict__ out_i,
                                                  const float* __restrict__ grad_out_t, double* __restrict__ mu,
                                                  double* __restrict__ musum)
{
    const size_t gtid = (size_t)blockIdx.x * blockDim.x + threadIdx.x, gs = (size_t)gridDim.x * blockDim.x;
    for (size_t x = gtid; x < nW; x += gs) {
        gw[x] = 0;
        gd[x] = 0;
    }
    for (size_t x = gtid; x < nT; x += gs) gt[x] = 0;
    if (gtid == 0) *wmax = 0u;
    for (size_t idx = gtid; idx < nn; idx += gs) {
        const int ns = min(out_n[idx], m.s_max);
        const size_t o = idx * (size_t)m.s_max;
        musum[idx] = spike_adjoints(m, ns, out_t + o, out_i + o, grad_out_t + o, mu + o);
    }
}

// max |w| over W^T: float bits of non-negative values order like the values,
// so an integer atomicMax gives the (order-free) maximum; one per workgroup
// (a few hundred workgroups at most), the waves' maxima joined in LDS.
constexpr int kWmaxBlocks = 256;

__global__ __launch_bounds__(256) void k_dly_wmax(const float* __restrict__ WT, size_t nW,
                                                 uint32_t* __restrict__ wmax)
{
    __shared__ float s_m[256 / kWave];
    const size_t gtid = (size_t)blockIdx.x * blockDim.x + threadIdx.x, gs = (size_t)gridDim.x * blockDim.x;
    float mx = 0.0f;
    for (size_t x = gtid; x < nW; x += gs) mx = fmaxf(mx, fabsf(WT[x]));
    for (int off = kWave / 2; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, kWave));
    if (threadIdx.x % kWave == 0) s_m[threadIdx.x / kWave] = mx;
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < 256 / kWave; ++w) mx = fmaxf(mx, s_m[w]);
        atomicMax(wmax, __float_as_uint(mx));
    }
}

// Fixed-point scales (one workgroup).  With M = max over neurons of
// sum_s |mu_s| (a bound of |P^m| and |P^s|, up to the e^{+ulp} of a spike
// time rounded below an arrival, which the extra bit of headroom covers),
// a contribution to dL/dw is at most 2 kappa M, one to dL/dd or dL/dt at most
// |w|max kappa M (1/tm + 1/ts); an element of dL/dW or dL/dD sums at most one
// per event of the batch, one of dL/dt one per neuron.  scale =
// 2^(61 - ceil(log2 bound)).
constexpr int kDlyScaleThreads = 1024;

__global__ __launch_bounds__(kDlyScaleThreads) void k_dly_scale(const double* __restrict__ musum, size_t nn,
                                                                const int32_t* __restrict__ ev_n, int B, int E_max,
                                                                int N, Model m, const uint32_t* __restrict__ wmax,
                                                                double* __restrict__ scale)
{
    __shared__ double s_max[kDlyScaleThreads];
    __shared__ double s_ev[kDlyScaleThreads];
    double mx = 0.0, ev = 0.0;
    for (size_t i = threadIdx.x; i < nn; i += kDlyScaleThreads) mx = fmax(mx, musum[i]);
    for (int b = threadIdx.x; b < B; b += kDlyScaleThreads) ev += (double)clamp_count(ev_n[b], E_max);
    s_max[threadIdx.x] = mx;
    s_ev[threadIdx.x] = ev;
    __syncthreads();
    for (int off = kDlyScaleThreads / 2; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off) {
            s_max[threadIdx.x] = fmax(s_max[threadIdx.x], s_max[threadIdx.x + off]);
            s_ev[threadIdx.x] += s_ev[threadIdx.x + off];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const double M = s_max[0], E = fmax(s_ev[0], 1.0), w = (double)__uint_as_float(*wmax);
        const double bw = 2.0 * m.kappa * M * E;
        const double bd = w * m.kappa * M * (m.inv_tm + m.inv_ts) * E;
        const double bt = w * m.kappa * M * (m.inv_tm + m.inv_ts) * (double)N;
        const double bounds[3] = {bw, bd, bt};
        for (int q = 0; q < 3; ++q) {
            int ex = 0;
            if (bounds[q] > 0.0 && isfinite(bounds[q])) frexp(bounds[q], &ex);   // bound < 2^ex
            scale[q] = ldexp(1.0, 61 - ex);
        }
    }
}

constexpr int kDlyWaves = 4;

__device__ __forceinline__ void fx_add(long long* p, double v, double sc)
{
    atomicAdd((unsigned long long*)p, (unsigned long long)llrint(v * sc));
}

// The walk of one (sample, neuron) item; add_wd(j, dL/dw_j, dL/dd_j) takes
// the weight and delay terms of an event from input channel j.
template <class AddWD>
__device__ __forceinline__ void dly_walk(size_t item, const float* __restrict__ q_t, const int32_t* __restrict__ q_k,
                                         const int32_t* __restrict__ ev_src, const int32_t* __restrict__ ev_n,
                                         int E_max, const float* __restrict__ WT, int C_in, int N, const Model& m,
                                         const float* __restrict__ out_t, const int32_t* __restrict__ out_n,
                                         const int32_t* __restrict__ out_k, const double* __restrict__ mu,
                                         const double* __restrict__ musum, const double* __restrict__ scale,
                                         AddWD add_wd, long long* __restrict__ tq, int32_t* __restrict__ tcnt)
{
    const int lane = (int)threadIdx.x % kWave;
    // spikes whose adjoints are all 0 add exactly 0 everywhere: not walked
    // (a NaN sum keeps them)
    const int ns = musum[item] == 0.0 ? 0 : min(out_n[item], m.s_max);
    const int b = (int)(item / (size_t)N), n = (int)(item % (size_t)N);
    const int nb = clamp_count(ev_n[b], E_max);
    const size_t so = item * (size_t)m.s_max;
    const float* st = out_t + so;
    const int32_t* sk = out_k + so;
    const double* mo = mu + so;
    const int klast = ns > 0 ? min(max(sk[ns - 1], 0), nb) : 0;   // queue events 0 .. klast - 1 feed a spike
    if (tcnt && lane == 0) tcnt[item] = klast;          // and get a dL/dt term in tq
    if (klast <= 0) return;
    long long* tqr = tq ? tq + item * (size_t)E_max : nullptr;
    const float* qa = q_t + item * (size_t)E_max;
    const int32_t* qi = q_k + item * (size_t)E_max;
    const int32_t* src = ev_src + (size_t)b * E_max;
    const double sT = scale[2];
    // the step holding queue event klast - 1, and the carry of the spikes
    // after it (every spike with out_k = klast), referred to its arrival
    int r_last = klast - 1;
    int f = (r_last / kWave) * kWave;
    double a_ref = (double)qa[r_last];
    int s_hi = ns;
    while (s_hi > 0 && sk[s_hi - 1] > r_last) --s_hi;
    double Cm = 0.0, Cs = 0.0;
    for (int s = s_hi + lane; s < ns; s += kWave) {
        const double u = fmax((double)st[s] - a_ref, 0.0);
        Cm += mo[s] * exp(-u * m.inv_tm);
        Cs += mo[s] * exp(-u * m.inv_ts);
    }
    for (int off = 1; off < kWave; off <<= 1) {
        Cm += __shfl_xor(Cm, off, kWave);
        Cs += __shfl_xor(Cs, off, kWave);
    }
    for (;;) {
        // spikes [s_lo, s_hi) have f < out_k <= r_last: after some event of the step
        int s_lo = s_hi;
        while (s_lo > 0 && sk[s_lo - 1] > f) --s_lo;
        const int e = f + lane;
        if (e <= r_last) {
            const double a = (double)qa[e];
            const int k = min(max(qi[e], 0), nb - 1);
            const int j = clamp_src(src[k], C_in);
            const double w = (double)WT[(size_t)j * N + n];
            double Pm = Cm * exp(-(a_ref - a) * m.inv_tm), Ps = Cs * exp(-(a_ref - a) * m.inv_ts);
            for (int s = s_lo; s < s_hi; ++s) {
                if (e < sk[s]) {
                    const double u = fmax((double)st[s] - a, 0.0);
                    Pm += mo[s] * exp(-u * m.inv_tm);
                    Ps += mo[s] * exp(-u * m.inv_ts);
                }
            }
            const double ga = w * m.kappa * (Pm * m.inv_tm - Ps * m.inv_ts);
            add_wd(j, m.kappa * (Pm - Ps), ga);
            if (tqr) tqr[e] = llrint(ga * sT);
        }
        if (f == 0) break;
        // the carry moved to the previous step's last event
        const double a2 = (double)qa[f - 1];
        Cm *= exp(-(a_ref - a2) * m.inv_tm);
        Cs *= exp(-(a_ref - a2) * m.inv_ts);
        for (int s = s_lo; s < s_hi; ++s) {
            const double u = fmax((double)st[s] - a2, 0.0);
            Cm += mo[s] * exp(-u * m.inv_tm);
            Cs += mo[s] * exp(-u * m.inv_ts);
        }
        a_ref = a2;
        r_last = f - 1;
        f -= kWave;
        s_hi = s_lo;
    }
}

// One wave per (sample, neuron); dL/dW and dL/dD added to global memory.
__global__ __launch_bounds__(kWave * kDlyWaves) void k_dly_adjoint(
    const float* __restrict__ q_t, const int32_t* __restrict__ q_k, const int32_t* __restrict__ ev_src,
    const int32_t* __restrict__ ev_n, int B, int E_max, const float* __restrict__ WT, int C_in, int N, Model m,
    const float* __restrict__ out_t, const int32_t* __restrict__ out_n, const int32_t* __restrict__ out_k,
    const double* __restrict__ mu, const double* __restrict__ musum, const double* __restrict__ scale,
    long long* __restrict__ gw, long long* __restrict__ gd, long long* __restrict__ tq, int32_t* __restrict__ tcnt)
{
    const size_t item = (size_t)blockIdx.x * kDlyWaves + threadIdx.x / kWave;
    if (item >= (size_t)B * N) return;
    const int n = (int)(item % (size_t)N);
    const double sW = scale[0], sD = scale[1];
    auto add_wd = [&](int j, double vw, double vd) {
        const size_t wi = (size_t)j * N + n;
        fx_add(&gw[wi], vw, sW);
        if (gd) fx_add(&gd[wi], vd, sD);
    };
    dly_walk(item, q_t, q_k, ev_src, ev_n, E_max, WT, C_in, N, m, out_t, out_n, out_k, mu, musum, scale, add_wd, tq,
             tcnt);
}

// For C_in <= kDlyLdsMaxC: one workgroup per (neuron, kDlyLdsWaves samples),
// a wave per sample; the neuron's dL/dW and dL/dD column is summed in LDS
// (2 C_in 64-bit fixed-point sums, order free) and added to global memory
// once per workgroup, nonzero entries only.
constexpr int kDlyLdsWaves = 8;
constexpr int kDlyLdsMaxC = 4096;

__global__ __launch_bounds__(kWave * kDlyLdsWaves) void k_dly_adjoint_lds(
    const float* __restrict__ q_t, const int32_t* __restrict__ q_k, const int32_t* __restrict__ ev_src,
    const int32_t* __restrict__ ev_n, int B, int E_max, const float* __restrict__ WT, int C_in, int N, Model m,
    const float* __restrict__ out_t, const int32_t* __restrict__ out_n, const int32_t* __restrict__ out_k,
    const double* __restrict__ mu, const double* __restrict__ musum, const double* __restrict__ scale,
    long long* __restrict__ gw, long long* __restrict__ gd, long long* __restrict__ tq, int32_t* __restrict__ tcnt,
    int nbg)
{
    extern __shared__ long long s_wd[];            // [C_in] dL/dW sums, then [C_in] dL/dD sums
    long long* s_w = s_wd;
    long long* s_d = s_wd + C_in;
    const int n = (int)(blockIdx.x / (unsigned)nbg), bg = (int)(blockIdx.x % (unsigned)nbg);
    const int tid = (int)threadIdx.x;
    for (int j = tid; j < C_in; j += (int)blockDim.x) {
        s_w[j] = 0;
        s_d[j] = 0;
    }
    __syncthreads();
    const int b = bg * kDlyLdsWaves + tid / kWave;
    if (b < B) {
        const double sW = scale[0], sD = scale[1];
        const bool want_d = gd != nullptr;
        auto add_wd = [&](int j, double vw, double vd) {
            atomicAdd((unsigned long long*)&s_w[j], (unsigned long long)llrint(vw * sW));
            if (want_d) atomicAdd((unsigned long long*)&s_d[j], (unsigned long long)llrint(vd * sD));
        };
        dly_walk((size_t)b * N + n, q_t, q_k, ev_src, ev_n, E_max, WT, C_in, N, m, out_t, out_n, out_k, mu, musum,
                 scale, add_wd, tq, tcnt);
    }
    __syncthreads();
    for (int j = tid; j < C_in; j += (int)blockDim.x) {
        const size_t wi = (size_t)j * N + n;
        const long long vw = s_w[j], vd = s_d[j];
        if (vw) atomicAdd((unsigned long long*)&gw[wi], (unsigned long long)vw);
        if (gd && vd) atomicAdd((unsigned long long*)&gd[wi], (unsigned long long)vd);
    }
}

// Fixed point -> float32 gradients.
__global__ __launch_bounds__(256) void k_dly_convert(const long long* __restrict__ gw,
                                                    const long long* __restrict__ gd,
                                                    const long long* __restrict__ gt,
                                                    const double* __restrict__ scale, size_t nW, size_t nT,
                                                    float* __restrict__ grad_WT, float* __restrict__ grad_DT,
                                                    float* __restrict__ grad_ev_t)
{
    const size_t gtid = (size_t)blockIdx.x * blockDim.x + threadIdx.x, gs = (size_t)gridDim.x * blockDim.x;
    const double iW = 1.0 / scale[0], iD = 1.0 / scale[1], iT = 1.0 / scale[2];
    for (size_t x = gtid; x < nW; x += gs) {
        grad_WT[x] = (float)((double)gw[x] * iW);
        if (grad_DT) grad_DT[x] = (float)((double)gd[x] * iD);
    }
    if (grad_ev_t)
        for (size_t x = gtid; x < nT; x += gs) grad_ev_t[x] = (float)((double)gt[x] * iT);
}

// dL/dt from the walks' per-event terms.  A walk stores the 64-bit
// fixed-point dL/dt term of each of its first tcnt[item] queue events at
// tq[item * stride + r] instead of adding it to dL/dt_k itself (every neuron
// of a sample adds to the same k, which makes those adds the walk's
// bottleneck).  One workgroup per (sample, group of neurons, range of kChunk
// event indices) sums its group's terms into LDS by event index (integer adds,
// order free) and adds each nonzero sum to gt once.
constexpr int kGtTargetBlocks = 1024;   // workgroups the neuron groups aim for

template <int kChunk, int kThreads>
__global__ __launch_bounds__(kThreads) void k_gt_gather(const int32_t* __restrict__ q_k,
                                                       const int32_t* __restrict__ ev_n,
                                                       const int32_t* __restrict__ tcnt, const long long* tq,
                                                       size_t stride, int E_max, int N, int ng, int nck,
                                                       long long* __restrict__ gt)
{
    __shared__ long long s_gt[kChunk];
    constexpr int kU = 4;                   // entries per thread in flight
    const int tid = (int)threadIdx.x;
    const int ck = (int)(blockIdx.x % (unsigned)nck);
    const int g = (int)((blockIdx.x / (unsigned)nck) % (unsigned)ng);
    const int b = (int)(blockIdx.x / ((unsigned)nck * (unsigned)ng));
    const int nb = clamp_count(ev_n[b], E_max);
    const int k0 = ck * kChunk, k1 = min(k0 + kChunk, nb);
    if (k0 >= k1) return;
    for (int i = tid; i < k1 - k0; i += kThreads) s_gt[i] = 0;
    __syncthreads();
    const int per = (N + ng - 1) / ng, n0 = g * per, n1 = min(N, n0 + per);
    for (int n = n0; n < n1; ++n) {
        const size_t item = (size_t)b * N + n;
        const int c = min(max(tcnt[item], 0), nb);
        const int32_t* qk = q_k + item * (size_t)E_max;
        const long long* tv = tq + item * stride;
        for (int r0 = 0; r0 < c; r0 += kU * kThreads) {
            int kk[kU];
            long long vv[kU];
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int r = r0 + u * kThreads + tid;
                const bool o = r < c;
                kk[u] = o ? min(max(qk[r], 0), nb - 1) : -1;
                vv[u] = o ? tv[r] : 0;
            }
#pragma unroll
            for (int u = 0; u < kU; ++u)
                if (vv[u] != 0 && kk[u] >= k0 && kk[u] < k1)
                    atomicAdd((unsigned long long*)&s_gt[kk[u] - k0], (unsigned long long)vv[u]);
        }
    }
    __syncthreads();
    for (int i = tid; i < k1 - k0; i += kThreads) {
        const long long v = s_gt[i];
        if (v) atomicAdd((unsigned long long*)&gt[(size_t)b * E_max + k0 + i], (unsigned long long)v);
    }
}

static void launch_gt_gather(const int32_t* q_k, const int32_t* ev_n, const int32_t* tcnt, const long long* tq,
                             size_t stride, int B, int E_max, int N, long long* gt, hipStream_t stream)
{
    if (B <= 0 || E_max <= 0) return;
    auto groups = [&](int nck) {
        const long long per_b = (long long)B * nck;
        long long ng = (kGtTargetBlocks + per_b - 1) / per_b;
        return (int)(ng < 1 ? 1 : (ng > N ? N : ng));
    };
    if (E_max <= 4096) {
        const int ng = groups(1);
        TIMED_LAUNCH("gt_gather", (k_gt_gather<4096, 256>), dim3((unsigned)((size_t)B * ng)), dim3(256), 0, stream,
                     q_k, ev_n, tcnt, tq, stride, E_max, N, ng, 1, gt);
    } else {
        const int nck = (E_max + 16383) / 16384;
        const int ng = groups(nck);
        TIMED_LAUNCH("gt_gather", (k_gt_gather<16384, 1024>), dim3((unsigned)((size_t)B * ng * nck)), dim3(1024), 0,
                     stream, q_k, ev_n, tcnt, tq, stride, E_max, N, ng, nck, gt);
    }
}

// ---------------------------------------------------------------------------
// Spike-count regularisers (App. E.1) of a layer with synaptic delays.  A
// neuron's input intervals lie between consecutive arrivals of its own queue
// (interval r ends at queue event r; interval nb is the open one up to
// t_end), so the walks run per (sample, neuron), one wave each, 64 queue
// events per step with lane l on event f + l and the interval it closes.
//   k_dreg_walk   forward: the event maps (decays from the arrival gaps, the
//                 weight jump) composed across the lanes by a log-depth scan
//                 give each interval's no-reset start state from the step's
//                 carried state; the reset deficit of the neuron's spikes is
//                 the carried deficit decayed by the same products plus the
//                 spikes of the step; V_max (reg_vmax_arg), the hinge sums and
//                 counts, and the per-interval record.
//   k_dregg_walk  backward: P_r = sum of the pseudo-spikes of the intervals
//                 after event r (mu e^{-(argmax - a_r)/tm}, and with ts), by
//                 P_{r-1} = A_r P_r + mu_r e^{-u_r/tm}: a suffix scan across
//                 the lanes from the carried P at the step's last event.  Per
//                 event dL/dw += kappa (P^m - P^s), dL/da = w kappa (P^m/tm -
//                 P^s/ts) plus the end-point slope terms, added to dL/dd and
//                 dL/dt; each spike's upstream gradient
//                 -((th - vr)/tm) P^m e^{-(a_r - t_s)/tm} at the event r that
//                 closes its interval.
// ---------------------------------------------------------------------------
constexpr int kDRegWaves = 4;

__global__ __launch_bounds__(kWave * kDRegWaves) void k_dreg_walk(
    const float* __restrict__ q_t, const int32_t* __restrict__ q_k, const int32_t* __restrict__ ev_src,
    const int32_t* __restrict__ ev_n, int B, int E_max, const float* __restrict__ WT, int C_in, int N, Model m,
    const float* __restrict__ out_t, const int32_t* __restrict__ out_n, const int32_t* __restrict__ out_k,
    double* __restrict__ ub, double* __restrict__ ob, float* __restrict__ under, float* __restrict__ over,
    double2* __restrict__ counts, double* __restrict__ vpmax, float2* __restrict__ rec)
{
    const int lane = (int)threadIdx.x % kWave;
    // wave-uniform (scalar registers): the neuron's spike list is read with
    // scalar loads, which do not wait behind the queue loads in flight
    const size_t item = (size_t)__builtin_amdgcn_readfirstlane((int)(blockIdx.x * kDRegWaves + threadIdx.x / kWave));
    if (item >= (size_t)B * N) return;
    const int b = (int)(item / (size_t)N), n = (int)(item % (size_t)N);
    const int nb = clamp_count(ev_n[b], E_max);
    const float* qa = q_t + item * (size_t)E_max;
    const int32_t* qi = q_k + item * (size_t)E_max;
    const int32_t* src = ev_src + (size_t)b * E_max;
    const int ns = max(min(out_n[item], m.s_max), 0);
    const float* st = out_t + item * (size_t)m.s_max;
    const int32_t* sk = out_k + item * (size_t)m.s_max;
    float2* rb = rec ? rec + item * ((size_t)E_max + 1) : nullptr;
    double su = 0.0, so = 0.0, nsil = 0.0, nspk = 0.0, vpm = 0.0;
    auto take = [&](int j, double V0, double I0, double L, double A, double D, bool spiked, bool end_input) {
        const RegArg ra = reg_vmax_arg(m, V0, I0, L, A, D);
        const double vmax = ra.vmax;
        if (spiked) {
            so += fmax(vmax - m.th, 0.0);
            nspk += 1.0;
        } else {
            su += fmax(m.th - vmax, 0.0);
            nsil += 1.0;
        }
        if (rb) {
            const float sgn = spiked ? (vmax > m.th ? -1.0f : 0.0f) : (vmax < m.th ? 1.0f : 0.0f);
            double slope = 0.0;
            if (ra.at_start) {
                slope = j > 0 ? (I0 - V0) * m.inv_tm : 0.0;
                rb[j] = make_record(sgn, kRecStart, 1.0, 1.0, slope);
            } else if (ra.at_end && end_input) {
                slope = (I0 * D - vmax) * m.inv_tm;
                rb[j] = make_record(sgn, kRecEnd, A, D, slope);
            } else {                             // inside, or the end t_end of the open interval
                rb[j] = make_record(sgn, kRecInside, ra.em, ra.es, 0.0);
            }
            if (sgn != 0.0f) vpm = fmax(vpm, fabs(slope));
        }
    };
    double U = 0.0, J = 0.0;       // no-reset state after event f - 1
    double Dc = 0.0;               // reset deficit there, of the spikes with out_k < f
    double a_prev = 0.0;           // arrival of event f - 1 (0 before the first)
    int sp = 0;                    // first spike with out_k >= f
    // The queue's loads run ahead of the walk: at step f the weights of step
    // f + 64 (their sources loaded a step earlier), the sources of step
    // f + 128 and the arrivals and event indices of step f + 192 are issued
    // before the step's work.
    auto ld_q = [&](int ff, float& a_, int& k_) {
        const int rr = ff + lane;
        const bool o = rr < nb;
        a_ = o ? qa[rr] : 0.0f;
        k_ = o ? min(max(qi[rr], 0), nb - 1) : 0;
    };
    auto ld_j = [&](int k_) { return clamp_src(src[k_], C_in); };
    auto ld_w = [&](int ff, int j_) { return ff + lane < nb ? WT[(size_t)j_ * (size_t)N + n] : 0.0f; };
    float a0 = 0.0f, a1 = 0.0f, a2 = 0.0f, w0 = 0.0f;
    int k0 = 0, k1 = 0, k2 = 0, j1 = 0;
    if (nb > 0) {
        ld_q(0, a0, k0);
        w0 = ld_w(0, ld_j(k0));
        ld_q(kWave, a1, k1);
        j1 = ld_j(k1);
        ld_q(2 * kWave, a2, k2);
    }
    for (int f = 0; f < nb; f += kWave) {
        const int r = f + lane;
        const bool ok = r < nb;
        const int lv = min(kWave - 1, nb - 1 - f);          // the step's last event (lane)
        const float w1 = ld_w(f + kWave, j1);
        const int j2 = ld_j(k2);
        float a3;
        int k3;
        ld_q(f + 3 * kWave, a3, k3);
        const float af = a0, w = w0;
        a0 = a1;
        w0 = w1;
        a1 = a2;
        j1 = j2;
        a2 = a3;
        k2 = k3;
        double ap = __shfl_up((double)af, 1, kWave);         // arrival of event r - 1
        if (lane == 0) ap = a_prev;
        const double a = (double)af;
        const double L = a - ap;
        double A = 1.0, D = 1.0;
        if (ok) {
            A = exp(-L * m.inv_tm);
            D = exp(-L * m.inv_ts);
        }
        double aU = A, bU = ok ? (double)w : 0.0, aJ = D, bJ = bU;
        scan_maps_up(aU, bU, lane);
        scan_maps_up(aJ, bJ, lane);
        double eaU = __shfl_up(aU, 1, kWave), ebU = __shfl_up(bU, 1, kWave);
        double eaJ = __shfl_up(aJ, 1, kWave), ebJ = __shfl_up(bJ, 1, kWave);
        if (lane == 0) {
            eaU = 1.0;
            ebU = 0.0;
            eaJ = 1.0;
            ebJ = 0.0;
        }
        const double U0 = fma(eaU, U, ebU), J0 = fma(eaJ, J, ebJ);     // at interval r's start
        // the deficit at interval r's start: the carried one decayed over
        // events f .. r - 1 (the product eaU), plus the spikes of intervals
        // f .. r - 1
        double Dft = Dc * eaU;
        bool spiked = false;
        for (int s = sp; s < ns && sk[s] < f + kWave; ++s) {
            const int ks = sk[s];
            if (ks < r) Dft += m.dth * exp(-(ap - (double)st[s]) * m.inv_tm);
            spiked |= ks == r;
        }
        if (ok) take(r, v_of(m, U0, J0) - Dft, J0, L, A, D, spiked, true);
        // the carry: the state after the step's last event, its arrival and
        // the deficit there
        const double Un = fma(aU, U, bU), Jn = fma(aJ, J, bJ);
        const double a_last = __shfl(a, lv, kWave);
        double Dn = Dc * __shfl(aU, lv, kWave);
        while (sp < ns && sk[sp] <= f + lv) {
            Dn += m.dth * exp(-(a_last - (double)st[sp]) * m.inv_tm);
            ++sp;
        }
        U = __shfl(Un, lv, kWave);
        J = __shfl(Jn, lv, kWave);
        Dc = Dn;
        a_prev = a_last;
    }
    {
        // the open interval after the last arrival, up to t_end
        const double L = m.t_end - a_prev;
        const double A = isinf(L) ? 0.0 : exp(-L * m.inv_tm), D = isinf(L) ? 0.0 : exp(-L * m.inv_ts);
        bool spiked = false;
        for (int s = sp; s < ns; ++s) spiked |= sk[s] == nb;
        if (lane == 0) take(nb, v_of(m, U, J) - Dc, J, L, A, D, spiked, false);
    }
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        su += __shfl_xor(su, off, kWave);
        so += __shfl_xor(so, off, kWave);
        nsil += __shfl_xor(nsil, off, kWave);
        nspk += __shfl_xor(nspk, off, kWave);
        vpm = fmax(vpm, __shfl_xor(vpm, off, kWave));
    }
    if (lane == 0) {
        const double u = nsil > 0.0 ? su / nsil : 0.0;
        const double o = nspk > 0.0 ? so / nspk : 0.0;
        ub[item] = u;
        ob[item] = o;
        if (under) under[item] = (float)u;
        if (over) over[item] = (float)o;
        if (counts) counts[item] = make_double2(nsil, nspk);
        if (vpmax) vpmax[item] = vpm;
    }
}

// Fixed-point scales of the delayed regularisers' gradient (one workgroup):
// M = the largest |G_u| nsil + |G_o| nspk (a bound of |P|), Gm the largest
// |G|, Vp the largest end-point slope of an active record.  A dL/dw term is
// at most 2 kappa M; a dL/da term at most w_max kappa M (1/tm + 1/ts) +
// 2 Gm Vp; dL/dW and dL/dD sum at most one term per event of the batch, dL/dt
// one per neuron: scale = 2^(61 - ceil(log2(bound))) each.
__global__ __launch_bounds__(kDlyScaleThreads) void k_dregg_scale(const double* __restrict__ musum,
                                                                const double2* __restrict__ coef,
                                                                const double* __restrict__ vpmax, size_t nn,
                                                                const int32_t* __restrict__ ev_n, int B, int E_max,
                                                                int N, Model m, const uint32_t* __restrict__ wmax,
                                                                double* __restrict__ scale)
{
    __shared__ double s_m[kDlyScaleThreads], s_g[kDlyScaleThreads], s_v[kDlyScaleThreads], s_e[kDlyScaleThreads];
    double M = 0.0, Gm = 0.0, Vp = 0.0, ev = 0.0;
    for (size_t i = threadIdx.x; i < nn; i += kDlyScaleThreads) {
        M = fmax(M, musum[i]);
        Gm = fmax(Gm, fmax(fabs(coef[i].x), fabs(coef[i].y)));
        Vp = fmax(Vp, vpmax[i]);
    }
    for (int b = threadIdx.x; b < B; b += kDlyScaleThreads) ev += (double)clamp_count(ev_n[b], E_max);
    s_m[threadIdx.x] = M;
    s_g[threadIdx.x] = Gm;
    s_v[threadIdx.x] = Vp;
    s_e[threadIdx.x] = ev;
    __syncthreads();
    for (int off = kDlyScaleThreads / 2; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off) {
            s_m[threadIdx.x] = fmax(s_m[threadIdx.x], s_m[threadIdx.x + off]);
            s_g[threadIdx.x] = fmax(s_g[threadIdx.x], s_g[threadIdx.x + off]);
            s_v[threadIdx.x] = fmax(s_v[threadIdx.x], s_v[threadIdx.x + off]);
            s_e[threadIdx.x] += s_e[threadIdx.x + off];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const double E = fmax(s_e[0], 1.0), w = (double)__uint_as_float(*wmax);
        const double term = w * m.kappa * s_m[0] * (m.inv_tm + m.inv_ts) + 2.0 * s_g[0] * s_v[0];
        const double bounds[3] = {2.0 * m.kappa * s_m[0] * E, term * E, term * (double)N};
        for (int q = 0; q < 3; ++q) {
            int ex = 0;
            if (bounds[q] > 0.0 && isfinite(bounds[q])) frexp(bounds[q], &ex);   // bound < 2^ex
            scale[q] = ldexp(1.0, 61 - ex);
        }
    }
}

// The backward walk of one (sample, neuron) item; add_wd(j, dL/dw_j,
// dL/dd_j) takes the weight and delay terms of an event from channel j.
template <class AddWD>
__device__ __forceinline__ void dregg_walk(size_t item, const float* __restrict__ q_t,
                                           const int32_t* __restrict__ q_k, const int32_t* __restrict__ ev_src,
                                           const int32_t* __restrict__ ev_n, int E_max, const float* __restrict__ WT,
                                           int C_in, int N, const Model& m, const float* __restrict__ out_t,
                                           const int32_t* __restrict__ out_n, const int32_t* __restrict__ out_k,
                                           float2* rec, const double2* __restrict__ coef,
                                           const double* __restrict__ scale, AddWD add_wd,
                                           int32_t* __restrict__ tcnt, float* __restrict__ grad_spike)
{
    const int lane = (int)threadIdx.x % kWave;
    const int b = (int)(item / (size_t)N), n = (int)(item % (size_t)N);
    const int nb = clamp_count(ev_n[b], E_max);
    const double2 G = coef[item];
    const bool live = nb > 0 && (G.x != 0.0 || G.y != 0.0);
    if (tcnt && lane == 0) tcnt[item] = live ? nb : 0;  // queue events with a dL/dt term
    if (!live) return;
    const float* qa = q_t + item * (size_t)E_max;
    const int32_t* qi = q_k + item * (size_t)E_max;
    const int32_t* src = ev_src + (size_t)b * E_max;
    const int ns = max(min(out_n[item], m.s_max), 0);
    const float* st = out_t + item * (size_t)m.s_max;
    const int32_t* sk = out_k + item * (size_t)m.s_max;
    float* gsp = grad_spike + item * (size_t)m.s_max;
    // the item's records; with tcnt, record r is overwritten by the 64-bit
    // fixed-point dL/dt term of queue event r once the walk has read it
    // (three steps before), stored as a float2 of the same bits
    float2* rb = rec + item * ((size_t)E_max + 1);
    const double sT = scale[2], kap = m.kappa, skp = -(m.dth * m.inv_tm);
    // P at event nb - 1: the open interval's pseudo-spike; tn: that interval
    RecTerm tn = rec_term(rb[nb], G, 0.0, 0.0);
    double Pm = tn.mu * tn.em, Ps = tn.mu * tn.es;
    int s_hi = ns;                                        // spikes with out_k <= the step's last event
    while (s_hi > 0 && sk[s_hi - 1] > nb - 1) --s_hi;
    // The queue's loads run ahead of the walk (steps going down): at step f
    // the weights of step f - 64 (their sources loaded a step earlier), the
    // sources of step f - 128 and the arrivals, event indices and records of
    // step f - 192 are issued before the step's work.
    auto ld_q = [&](int ff, float& a_, int& k_, float2& rc_) {
        const int rr = ff + lane;
        const bool o = ff >= 0 && rr < nb;
        a_ = o ? qa[rr] : 0.0f;
        k_ = o ? min(max(qi[rr], 0), nb - 1) : 0;
        rc_ = o ? rb[rr] : make_float2(0.0f, 0.0f);
    };
    auto ld_j = [&](int k_) { return clamp_src(src[k_], C_in); };
    auto ld_w = [&](int ff, int j_) { return ff >= 0 && ff + lane < nb ? WT[(size_t)j_ * (size_t)N + n] : 0.0f; };
    const int ftop = ((nb - 1) / kWave) * kWave;
    float a0, a1, a2, w0;
    int k0, k1, k2, j0, j1;
    float2 c0, c1, c2;
    ld_q(ftop, a0, k0, c0);
    j0 = ld_j(k0);
    w0 = ld_w(ftop, j0);
    ld_q(ftop - kWave, a1, k1, c1);
    j1 = ld_j(k1);
    ld_q(ftop - 2 * kWave, a2, k2, c2);
    for (int f = ftop; f >= 0; f -= kWave) {
        const int r = f + lane;
        const bool ok = r < nb;
        const int hi = min(f + kWave - 1, nb - 1);
        const float w1 = ld_w(f - kWave, j1);
        const int j2 = ld_j(k2);
        float a3;
        int k3;
        float2 c3;
        ld_q(f - 3 * kWave, a3, k3, c3);
        const float af = a0;
        const int j = j0;
        const double w = ok ? (double)w0 : 0.0;
        const float2 rc = c0;
        // the arrival before each event: the lane below, or the step below's last
        const double ap = wave_shr1((double)af, f > 0 ? read_lane_double((double)a1, kWave - 1) : 0.0);
        a0 = a1; k0 = k1; j0 = j1; w0 = w1; c0 = c1;
        a1 = a2; k1 = k2; j1 = j2; c1 = c2;
        a2 = a3; k2 = k3; c2 = c3;
        const double a = (double)af;
        double A = 1.0, D = 1.0;
        RecTerm t{0.0, 0.0, 0.0, 0.0, 0.0};
        if (ok) {
            const double L = a - ap;
            A = exp(-L * m.inv_tm);
            D = exp(-L * m.inv_ts);
            t = rec_term(rc, G, A, D);                    // interval r, closed by event r
        }
        // the record after event r: lane r + 1's, or the carried one at the top
        RecTerm tx;
        tx.mu = wave_shl1(t.mu, 0.0);
        tx.vs = wave_shl1(t.vs, 0.0);
        if (r == hi) {
            tx.mu = tn.mu;
            tx.vs = tn.vs;
        }
        // P at event r: the maps of lanes r + 1 .. hi applied to P at event hi
        double am = A, bm = t.mu * t.em, as = D, bs = t.mu * t.es;
        scan_maps_down(am, bm, lane);
        scan_maps_down(as, bs, lane);
        const double xam = wave_shl1(am, 1.0), xbm = wave_shl1(bm, 0.0);
        const double xas = wave_shl1(as, 1.0), xbs = wave_shl1(bs, 0.0);
        const double Pmr = fma(xam, Pm, xbm), Psr = fma(xas, Ps, xbs);
        if (ok) {
            double ga = w * kap * (Pmr * m.inv_tm - Psr * m.inv_ts);
            ga = fma(tx.mu, tx.vs, ga);                   // 0 unless that argmax is the interval's start
            ga = fma(t.mu, t.ve, ga);                     // 0 unless this argmax is the interval's end
            add_wd(j, kap * (Pmr - Psr), ga);
            if (tcnt) rb[r] = __builtin_bit_cast(float2, (long long)llrint(ga * sT));
        }
        // the spikes of intervals f .. hi: upstream gradient from P at the
        // event that closes their interval
        int s_lo = s_hi;
        while (s_lo > 0 && sk[s_lo - 1] >= f) --s_lo;
        for (int s = s_lo; s < s_hi; ++s)
            if (sk[s] == r) gsp[s] += (float)(skp * Pmr * exp(-(a - (double)st[s]) * m.inv_tm));
        // the carry: P at event f - 1 and the record of interval f
        Pm = read_lane_double(fma(am, Pm, bm), 0);
        Ps = read_lane_double(fma(as, Ps, bs), 0);
        tn.mu = read_lane_double(t.mu, 0);
        tn.vs = read_lane_double(t.vs, 0);
        s_hi = s_lo;
    }
}

// dL/dW and dL/dD to global memory (C_in > kDlyLdsMaxC).
__global__ __launch_bounds__(kWave * kDRegWaves) void k_dregg_walk(
    const float* __restrict__ q_t, const int32_t* __restrict__ q_k, const int32_t* __restrict__ ev_src,
    const int32_t* __restrict__ ev_n, int B, int E_max, const float* __restrict__ WT, int C_in, int N, Model m,
    const float* __restrict__ out_t, const int32_t* __restrict__ out_n, const int32_t* __restrict__ out_k,
    float2* rec, const double2* __restrict__ coef, const double* __restrict__ scale,
    long long* __restrict__ gw, long long* __restrict__ gd, int32_t* __restrict__ tcnt,
    float* __restrict__ grad_spike)
{
    const size_t item = (size_t)__builtin_amdgcn_readfirstlane((int)(blockIdx.x * kDRegWaves + threadIdx.x / kWave));
    if (item >= (size_t)B * N) return;
    const int n = (int)(item % (size_t)N);
    const double sW = scale[0], sD = scale[1];
    auto add_wd = [&](int j, double vw, double vd) {
        const size_t wi = (size_t)j * N + n;
        fx_add(&gw[wi], vw, sW);
        if (gd) fx_add(&gd[wi], vd, sD);
    };
    dregg_walk(item, q_t, q_k, ev_src, ev_n, E_max, WT, C_in, N, m, out_t, out_n, out_k, rec, coef, scale, add_wd,
               tcnt, grad_spike);
}

// C_in <= kDlyLdsMaxC: one workgroup per (neuron, kDlyLdsWaves samples), the
// neuron's dL/dW and dL/dD column summed in LDS as in k_dly_adjoint_lds.
__global__ __launch_bounds__(kWave * kDlyLdsWaves) void k_dregg_walk_lds(
    const float* __restrict__ q_t, const int32_t* __restrict__ q_k, const int32_t* __restrict__ ev_src,
    const int32_t* __restrict__ ev_n, int B, int E_max, const float* __restrict__ WT, int C_in, int N, Model m,
    const float* __restrict__ out_t, const int32_t* __restrict__ out_n, const int32_t* __restrict__ out_k,
    float2* rec, const double2* __restrict__ coef, const double* __restrict__ scale,
    long long* __restrict__ gw, long long* __restrict__ gd, int32_t* __restrict__ tcnt,
    float* __restrict__ grad_spike, int nbg)
{
    extern __shared__ long long s_wd[];            // [C_in] dL/dW sums, then [C_in] dL/dD sums
    long long* s_w = s_wd;
    long long* s_d = s_wd + C_in;
    const int n = (int)(blockIdx.x / (unsigned)nbg), bg = (int)(blockIdx.x % (unsigned)nbg);
    const int tid = (int)threadIdx.x;
    for (int j = tid; j < C_in; j += (int)blockDim.x) {
        s_w[j] = 0;
        s_d[j] = 0;
    }
    __syncthreads();
    const int b = __builtin_amdgcn_readfirstlane(bg * kDlyLdsWaves + tid / kWave);
    if (b < B) {
        const double sW = scale[0], sD = scale[1];
        const bool want_d = gd != nullptr;
        auto add_wd = [&](int j, double vw, double vd) {
            atomicAdd((unsigned long long*)&s_w[j], (unsigned long long)llrint(vw * sW));
            if (want_d) atomicAdd((unsigned long long*)&s_d[j], (unsigned long long)llrint(vd * sD));
        };
        dregg_walk((size_t)b * N + n, q_t, q_k, ev_src, ev_n, E_max, WT, C_in, N, m, out_t, out_n, out_k, rec, coef,
                   scale, add_wd, tcnt, grad_spike);
    }
    __syncthreads();
    for (int j = tid; j < C_in; j += (int)blockDim.x) {
        const size_t wi = (size_t)j * N + n;
        const long long vw = s_w[j], vd = s_d[j];
        if (vw) atomicAdd((unsigned long long*)&gw[wi], (unsigned long long)vw);
        if (gd && vd) atomicAdd((unsigned long long*)&gd[wi], (unsigned long long)vd);
    }
}

__global__ __launch_bounds__(256) void k_dregg_zero(size_t nW, size_t nT, long long* __restrict__ gw,
                                                   long long* __restrict__ gd, long long* __restrict__ gt,
                                                   uint32_t* __restrict__ wmax)
{
    const size_t gtid = (size_t)blockIdx.x * blockDim.x + threadIdx.x, gs = (size_t)gridDim.x * blockDim.x;
    for (size_t x = gtid; x < nW; x += gs) {
        gw[x] = 0;
        gd[x] = 0;
    }
    for (size_t x = gtid; x < nT; x += gs) gt[x] = 0;
    if (gtid == 0) *wmax = 0u;
}

static unsigned grid_for(size_t work)
{
    size_t blocks = (work + 255) / 256;
    if (blocks > 2048) blocks = 2048;
    if (blocks < 1) blocks = 1;
    return (unsigned)blocks;
}

}  // namespace lif

// Workspace of lif_delay_queues: the arrivals [B][N][E_max] (float), and
// for queues longer than kQLdsMax the binned keys (64-bit).
static void dly_queue_layout(int B, int E_max, int N, size_t& arr_bytes, size_t& key_bytes)
{
    const size_t n = (size_t)B * (size_t)N * (size_t)E_max;
    arr_bytes = (n * sizeof(float) + 255) & ~(size_t)255;
    key_bytes = E_max > lif::kQLdsMax ? (n * sizeof(unsigned long long) + 255) & ~(size_t)255 : 0;
}

extern "C" size_t lif_delay_queues_workspace_size(int B, int E_max, int N_out)
{
    if (B < 0 || E_max < 0 || N_out < 1) return 0;
    size_t arr_bytes, key_bytes;
    dly_queue_layout(B, E_max, N_out, arr_bytes, key_bytes);
    return arr_bytes + key_bytes + 256;
}

extern "C" int lif_delay_queues(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                                const float* DT, int C_in, int N_out, float* q_t, int32_t* q_k, int32_t* status,
                                void* ws, size_t ws_bytes, lif_stream_t stream_)
{
    using namespace lif;
    if (B < 0 || E_max < 0 || C_in < 1 || N_out < 1) return LIF_ERR_ARG;
    if (B > 0 && E_max > 0 && (!ev_t || !ev_src || !ev_n || !DT || !q_t || !q_k || !ws)) return LIF_ERR_ARG;
    if ((size_t)B * (size_t)N_out >= ((size_t)1 << 31) || B > 65535) return LIF_ERR_SIZE;
    if (ws_bytes < lif_delay_queues_workspace_size(B, E_max, N_out)) return LIF_ERR_WORKSPACE;
    hipStream_t stream = (hipStream_t)stream_;
    if (status) {
        TIMED_LAUNCH("dly_status_reset", k_dly_status_reset, dim3(1), dim3(kWave), 0, stream, status);
        const size_t nD = (size_t)C_in * N_out;
        TIMED_LAUNCH("dly_check", k_dly_check, dim3(grid_for(nD)), dim3(256), 0, stream, DT, nD, ev_n, B, E_max,
                     status);
    }
    if (B > 0 && E_max > 0) {
        size_t arr_bytes, key_bytes;
        dly_queue_layout(B, E_max, N_out, arr_bytes, key_bytes);
        float* arr = (float*)(((uintptr_t)ws + 255) & ~(uintptr_t)255);
        unsigned long long* keys = (unsigned long long*)((char*)arr + arr_bytes);
        const dim3 agrid((unsigned)((E_max + kArrTile - 1) / kArrTile), (unsigned)B,
                         (unsigned)((N_out + kArrTile - 1) / kArrTile));
        TIMED_LAUNCH("dly_arrival", k_dly_arrival, agrid, dim3(256), 0, stream, ev_t, ev_src, ev_n, E_max, DT, C_in,
                     N_out, arr);
        const dim3 qgrid((unsigned)((size_t)B * N_out));
        TIMED_LAUNCH("dly_queue", (k_dly_queue_lds<0, 8192, 512, 2048, 4>), qgrid, dim3(512), 0, stream, ev_n, E_max,
                     N_out, arr, q_t, q_k);
        if (E_max > 8192)
            TIMED_LAUNCH("dly_queue", (k_dly_queue_lds<8192, 11520, 768, 2048, 6>), qgrid, dim3(768), 0, stream,
                         ev_n, E_max, N_out, arr, q_t, q_k);
        if (E_max > 11520)
            TIMED_LAUNCH("dly_queue", (k_dly_queue_lds<11520, kQLdsMax, 1024, 4096, 4>), qgrid, dim3(1024), 0,
                         stream, ev_n, E_max, N_out, arr, q_t, q_k);
        if (E_max > kQLdsMax)
            TIMED_LAUNCH("dly_queue", k_dly_queue, qgrid, dim3(kQThreads), 0, stream, ev_n, E_max, N_out, arr, keys,
                         q_t, q_k);
    }
    return check_launch();
}

extern "C" int lif_layer_forward_delayed(const float* q_t, const int32_t* q_k, const int32_t* ev_src,
                                         const int32_t* ev_n, int B, int E_max, const float* WT, int C_in,
                                         int N_out, const lif_params* p, float* out_t, int32_t* out_n, float* out_i,
                                         int32_t* out_k, int32_t* status, lif_stream_t stream_)
{
    using namespace lif;
    int rc = validate_forward_args(q_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, p, out_t, out_n, status);
    if (rc) return rc;
    if (B > 0 && E_max > 0 && !q_k) return LIF_ERR_ARG;
    if ((size_t)B * (size_t)N_out >= ((size_t)1 << 31)) return LIF_ERR_SIZE;
    // no budget: a neuron stops when its queue is consumed or at s_max spikes
    return launch_chunked_walk(q_t, ev_src, ev_n, q_k, B, E_max, WT, C_in, N_out, make_model(*p), 128, 0x7fffffff,
                               out_t, out_n, out_i, out_k, nullptr, nullptr, status, (hipStream_t)stream_);
}

extern "C" int lif_layer_forward_delayed_sequential(const float* q_t, const int32_t* q_k, const int32_t* ev_src,
                                                    const int32_t* ev_n, int B, int E_max, const float* WT, int C_in,
                                                    int N_out, const lif_params* p, float* out_t, int32_t* out_n,
                                                    float* out_i, int32_t* out_k, int32_t* status,
                                                    lif_stream_t stream_)
{
    using namespace lif;
    int rc = validate_forward_args(q_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, p, out_t, out_n, status);
    if (rc) return rc;
    if (B > 0 && E_max > 0 && !q_k) return LIF_ERR_ARG;
    if ((size_t)B * (size_t)N_out >= ((size_t)1 << 31)) return LIF_ERR_SIZE;
    return launch_sequential_queue(q_t, q_k, ev_src, ev_n, B, E_max, WT, C_in, N_out, make_model(*p), out_t, out_n,
                                   out_i, out_k, status, (hipStream_t)stream_);
}

extern "C" size_t lif_layer_backward_delayed_workspace_size(int B, int E_max, int C_in, int N_out,
                                                            const lif_params* p)
{
    if (B < 0 || E_max < 0 || C_in < 1 || N_out < 1 || !p || p->s_max < 1) return 0;
    return lif::dly_bwd_layout(B, E_max, C_in, N_out, p->s_max, true).total;
}

extern "C" int lif_layer_backward_delayed(const float* q_t, const int32_t* q_k, const int32_t* ev_src,
                                          const int32_t* ev_n, int B, int E_max, const float* WT, int C_in,
                                          int N_out, const lif_params* p, const float* out_t, const int32_t* out_n,
                                          const float* out_i, const int32_t* out_k, const float* grad_out_t,
                                          float* grad_WT, float* grad_DT, float* grad_ev_t, void* ws,
                                          size_t ws_bytes, lif_stream_t stream_)
{
    using namespace lif;
    if (!p || !WT || !grad_WT || B < 0 || E_max < 0 || C_in < 1 || N_out < 1) return LIF_ERR_ARG;
    int rc = check_params(p);
    if (rc) return rc;
    if (B > 0 && (!ev_n || !out_t || !out_n || !out_i || !out_k || !grad_out_t)) return LIF_ERR_ARG;
    if (B > 0 && E_max > 0 && (!q_t || !q_k || !ev_src)) return LIF_ERR_ARG;
    if ((size_t)B * (size_t)N_out >= ((size_t)1 << 31)) return LIF_ERR_SIZE;
    const DlyBwdLayout L = dly_bwd_layout(B, E_max, C_in, N_out, p->s_max, grad_ev_t != nullptr);
    if (!ws || ws_bytes < L.total) return LIF_ERR_WORKSPACE;
    hipStream_t stream = (hipStream_t)stream_;
    const Model m = make_model(*p);
    char* base = (char*)(((uintptr_t)ws + 255) & ~(uintptr_t)255);
    double* mu = (double*)(base + L.mu);
    double* musum = (double*)(base + L.musum);
    double* scale = (double*)(base + L.scale);
    uint32_t* wmax = (uint32_t*)(base + L.wmax);
    long long* gw = (long long*)(base + L.gw);
    long long* gd = (long long*)(base + L.gd);
    long long* gt = (long long*)(base + L.gt);
    int32_t* tcnt = grad_ev_t ? (int32_t*)(base + L.tcnt) : nullptr;
    long long* tq = grad_ev_t ? (long long*)(base + L.tq) : nullptr;
    const size_t nW = (size_t)C_in * N_out, nT = (size_t)B * E_max, nn = (size_t)B * N_out;
    size_t work = nW > nT ? nW : nT;
    if (nn > work) work = nn;
    TIMED_LAUNCH("dly_setup", k_dly_setup, dim3(grid_for(work)), dim3(256), 0, stream, nW, nT, gw, gd, gt, wmax, nn,
                 m, out_t, out_n, out_i, grad_out_t, mu, musum);
    TIMED_LAUNCH("dly_wmax", k_dly_wmax, dim3(std::min(grid_for(nW), (unsigned)kWmaxBlocks)), dim3(256), 0, stream,
                 WT, nW, wmax);
    TIMED_LAUNCH("dly_scale", k_dly_scale, dim3(1), dim3(kDlyScaleThreads), 0, stream, musum, nn, ev_n, B, E_max,
                 N_out, m, wmax, scale);
    if (nn && E_max > 0) {
        if (C_in <= kDlyLdsMaxC) {
            const int nbg = (B + kDlyLdsWaves - 1) / kDlyLdsWaves;
            TIMED_LAUNCH("dly_adjoint", k_dly_adjoint_lds, dim3((unsigned)((size_t)N_out * nbg)),
                         dim3(kWave * kDlyLdsWaves), (size_t)2 * C_in * sizeof(long long), stream, q_t, q_k, ev_src, ev_n, B, E_max, WT, C_in, N_out, m,
                         out_t, out_n, out_k, mu, musum, scale, gw, grad_DT ? gd : nullptr, tq, tcnt, nbg);
        } else {
            TIMED_LAUNCH("dly_adjoint", k_dly_adjoint, dim3((unsigned)((nn + kDlyWaves - 1) / kDlyWaves)),
                         dim3(kWave * kDlyWaves), 0, stream, q_t, q_k, ev_src, ev_n, B, E_max, WT, C_in, N_out, m,
                         out_t, out_n, out_k, mu, musum, scale, gw, grad_DT ? gd : nullptr, tq, tcnt);
        }
        if (grad_ev_t) launch_gt_gather(q_k, ev_n, tcnt, tq, (size_t)E_max, B, E_max, N_out, gt, stream);
    }
    TIMED_LAUNCH("dly_convert", k_dly_convert, dim3(grid_for(work)), dim3(256), 0, stream, gw, gd, gt, scale, nW, nT,
                 grad_WT, grad_DT, grad_ev_t);
    return check_launch();
}

// ---------------------------------------------------------------------------
// Spike-count regularisers of a layer with synaptic delays
// ---------------------------------------------------------------------------
namespace lif {

struct DRegLayout {
    size_t ub, ob, counts, gates, coef, musum, vpmax, rec, wmax, scale, gw, gd, gt, tcnt, total;
};

static DRegLayout dreg_layout(int B, int E_max, int C_in, int N, bool grad)
{
    DRegLayout L{};
    size_t off = 0;
    auto take = [&](size_t bytes) { size_t o = off; off += (bytes + 255) & ~(size_t)255; return o; };
    const size_t nn = (size_t)B * N;
    L.ub = take(nn * sizeof(double));
    L.ob = take(nn * sizeof(double));
    L.counts = take(nn * sizeof(double2));
    L.gates = take((size_t)N * sizeof(double2));
    if (grad) {
        L.coef = take(nn * sizeof(double2));
        L.musum = take(nn * sizeof(double));
        L.vpmax = take(nn * sizeof(double));
        L.rec = take(nn * ((size_t)E_max + 1) * sizeof(float2));
        L.wmax = take(sizeof(uint32_t));
        L.scale = take(4 * sizeof(double));
        L.gw = take((size_t)C_in * N * sizeof(long long));
        L.gd = take((size_t)C_in * N * sizeof(long long));
        L.gt = take((size_t)B * E_max * sizeof(long long));
        L.tcnt = take(nn * sizeof(int32_t));
    }
    L.total = off + 256;
    return L;
}

static int dreg_check(const float* q_t, const int32_t* q_k, const int32_t* ev_src, const int32_t* ev_n, int B,
                      int E_max, const float* WT, int C_in, int N_out, const lif_params* p, const float* out_t,
                      const int32_t* out_n, const int32_t* out_k, double c_target)
{
    if (!p || !WT || B < 0 || E_max < 0 || C_in < 1 || N_out < 1) return LIF_ERR_ARG;
    int rc = check_params(p);
    if (rc) return rc;
    if (B > 0 && (!ev_n || !out_t || !out_n || !out_k)) return LIF_ERR_ARG;
    if (B > 0 && E_max > 0 && (!q_t || !q_k || !ev_src)) return LIF_ERR_ARG;
    if (!(c_target > 0.0) || !isfinite(c_target)) return LIF_ERR_ARG;
    if ((size_t)B * (size_t)N_out >= ((size_t)1 << 31) || B > 65535) return LIF_ERR_SIZE;
    return LIF_OK;
}

static void launch_dreg_walk(const float* q_t, const int32_t* q_k, const int32_t* ev_src, const int32_t* ev_n, int B,
                             int E_max, const float* WT, int C_in, int N, const Model& m, const float* out_t,
                             const int32_t* out_n, const int32_t* out_k, double* ub, double* ob, float* under,
                             float* over, double2* counts, double* vpmax, float2* rec, hipStream_t stream)
{
    const size_t nn = (size_t)B * N;
    if (nn == 0) return;
    TIMED_LAUNCH("dreg_walk", k_dreg_walk, dim3((unsigned)((nn + kDRegWaves - 1) / kDRegWaves)),
                 dim3(kWave * kDRegWaves), 0, stream, q_t, q_k, ev_src, ev_n, B, E_max, WT, C_in, N, m, out_t, out_n,
                 out_k, ub, ob, under, over, counts, vpmax, rec);
}

}  // namespace lif

extern "C" size_t lif_spike_count_reg_delayed_workspace_size(int B, int E_max, int C_in, int N_out)
{
    if (B < 0 || E_max < 0 || C_in < 1 || N_out < 1) return 0;
    return lif::dreg_layout(B, E_max, C_in, N_out, true).total;
}

extern "C" int lif_spike_count_reg_delayed(const float* q_t, const int32_t* q_k, const int32_t* ev_src,
                                           const int32_t* ev_n, int B, int E_max, const float* WT, int C_in,
                                           int N_out, const lif_params* p, const float* out_t, const int32_t* out_n,
                                           const int32_t* out_k, double c_target, float* loss, float* under,
                                           float* over, void* ws, size_t ws_bytes, lif_stream_t stream_)
{
    using namespace lif;
    int rc = dreg_check(q_t, q_k, ev_src, ev_n, B, E_max, WT, C_in, N_out, p, out_t, out_n, out_k, c_target);
    if (rc) return rc;
    const DRegLayout L = dreg_layout(B, E_max, C_in, N_out, false);
    if (!ws || ws_bytes < L.total) return LIF_ERR_WORKSPACE;
    hipStream_t stream = (hipStream_t)stream_;
    const Model m = make_model(*p);
    char* base = (char*)(((uintptr_t)ws + 255) & ~(uintptr_t)255);
    double* ub = (double*)(base + L.ub);
    double* ob = (double*)(base + L.ob);
    launch_dreg_walk(q_t, q_k, ev_src, ev_n, B, E_max, WT, C_in, N_out, m, out_t, out_n, out_k, ub, ob, under, over,
                     nullptr, nullptr, nullptr, stream);
    if (B > 0) launch_reg_loss(ub, ob, out_n, B, N_out, m.s_max, c_target, loss, nullptr, stream);
    return check_launch();
}

extern "C" int lif_spike_count_reg_delayed_backward(const float* q_t, const int32_t* q_k, const int32_t* ev_src,
                                                    const int32_t* ev_n, int B, int E_max, const float* WT, int C_in,
                                                    int N_out, const lif_params* p, const float* out_t,
                                                    const int32_t* out_n, const int32_t* out_k, double c_target,
                                                    double lam_reg, double lam_over, float* loss, float* grad_spike,
                                                    float* grad_WT, float* grad_DT, float* grad_ev_t, void* ws,
                                                    size_t ws_bytes, lif_stream_t stream_)
{
    using namespace lif;
    int rc = dreg_check(q_t, q_k, ev_src, ev_n, B, E_max, WT, C_in, N_out, p, out_t, out_n, out_k, c_target);
    if (rc) return rc;
    if (!grad_WT || (B > 0 && !grad_spike) || !isfinite(lam_reg) || !isfinite(lam_over)) return LIF_ERR_ARG;
    const DRegLayout L = dreg_layout(B, E_max, C_in, N_out, true);
    if (!ws || ws_bytes < L.total) return LIF_ERR_WORKSPACE;
    hipStream_t stream = (hipStream_t)stream_;
    const Model m = make_model(*p);
    char* base = (char*)(((uintptr_t)ws + 255) & ~(uintptr_t)255);
    double* ub = (double*)(base + L.ub);
    double* ob = (double*)(base + L.ob);
    double2* counts = (double2*)(base + L.counts);
    double2* gates = (double2*)(base + L.gates);
    double2* coef = (double2*)(base + L.coef);
    double* musum = (double*)(base + L.musum);
    double* vpmax = (double*)(base + L.vpmax);
    float2* rec = (float2*)(base + L.rec);
    uint32_t* wmax = (uint32_t*)(base + L.wmax);
    double* scale = (double*)(base + L.scale);
    long long* gw = (long long*)(base + L.gw);
    long long* gd = (long long*)(base + L.gd);
    long long* gt = (long long*)(base + L.gt);
    int32_t* tcnt = grad_ev_t ? (int32_t*)(base + L.tcnt) : nullptr;
    const size_t nW = (size_t)C_in * N_out, nT = (size_t)B * E_max, nn = (size_t)B * N_out;
    const size_t work = nW > nT ? nW : nT;
    TIMED_LAUNCH("dregg_zero", k_dregg_zero, dim3(grid_for(work)), dim3(256), 0, stream, nW, nT, gw, gd, gt, wmax);
    TIMED_LAUNCH("dly_wmax", k_dly_wmax, dim3(std::min(grid_for(nW), (unsigned)kWmaxBlocks)), dim3(256), 0, stream,
                 WT, nW, wmax);
    launch_dreg_walk(q_t, q_k, ev_src, ev_n, B, E_max, WT, C_in, N_out, m, out_t, out_n, out_k, ub, ob, nullptr,
                     nullptr, counts, vpmax, rec, stream);
    if (B > 0) {
        launch_reg_loss(ub, ob, out_n, B, N_out, m.s_max, c_target, loss, gates, stream);
        launch_regg_coef(counts, gates, out_n, B, N_out, m.s_max, c_target, lam_reg, lam_over, coef, musum, stream);
        TIMED_LAUNCH("dregg_scale", k_dregg_scale, dim3(1), dim3(kDlyScaleThreads), 0, stream, musum, coef, vpmax, nn,
                     ev_n, B, E_max, N_out, m, wmax, scale);
        if (E_max > 0) {
            if (C_in <= kDlyLdsMaxC) {
                const int nbg = (B + kDlyLdsWaves - 1) / kDlyLdsWaves;
                TIMED_LAUNCH("dregg_walk", k_dregg_walk_lds, dim3((unsigned)((size_t)N_out * nbg)),
                             dim3(kWave * kDlyLdsWaves), (size_t)2 * C_in * sizeof(long long), stream, q_t, q_k,
                             ev_src, ev_n, B, E_max, WT, C_in, N_out, m, out_t, out_n, out_k, rec, coef, scale, gw,
                             grad_DT ? gd : nullptr, tcnt, grad_spike, nbg);
            } else {
                TIMED_LAUNCH("dregg_walk", k_dregg_walk, dim3((unsigned)((nn + kDRegWaves - 1) / kDRegWaves)),
                             dim3(kWave * kDRegWaves), 0, stream, q_t, q_k, ev_src, ev_n, B, E_max, WT, C_in, N_out, m,
                             out_t, out_n, out_k, rec, coef, scale, gw, grad_DT ? gd : nullptr, tcnt,
                             grad_spike);
            }
            if (grad_ev_t)
                launch_gt_gather(q_k, ev_n, tcnt, (const long long*)rec, (size_t)E_max + 1, B, E_max, N_out, gt,
                                 stream);
        }
    } else {
        TIMED_LAUNCH("dregg_scale", k_dregg_scale, dim3(1), dim3(kDlyScaleThreads), 0, stream, musum, coef, vpmax,
                     (size_t)0, ev_n, 0, E_max, N_out, m, wmax, scale);
    }
    TIMED_LAUNCH("dly_convert", k_dly_convert, dim3(grid_for(work)), dim3(256), 0, stream, gw, gd, gt, scale, nW, nT,
                 grad_WT, grad_DT, grad_ev_t);
    return check_launch();
}
