// lif_merge.hip -- layer glue: the spikes of one layer become the next
// layer's sorted per-sample event queue (Appendix E.2: layerwise processing,
// spikes sorted into the queues of the next layer), and the first-spike
// softmax cross-entropy readout used to drive a backward pass.
//
// Merge: one workgroup per sample.  Each neuron's spikes are already in
// time order; the workgroup gathers them into LDS as 64-bit keys (float bits
// of the time, which order like the times since spike times are positive,
// then i * s_max + s, which orders equal times by neuron) and sorts them
// with a bitonic network in LDS, over the smallest power of two holding its
// keys (the LDS array is sized for the most a sample can hold).  When a
// sample has more spikes than the
// sort holds, the K = min(total, E2_max) earliest are found first: the
// K-th smallest time t_K by bisection on its float bits (each neuron's
// spikes are sorted, so counting the spikes at or before a time is a binary
// search per neuron), then every spike before t_K and, in neuron order, as
// many spikes at exactly t_K as K allows.
#include "lif_common.hpp"
#include "lif_host.hpp"

namespace lif {

constexpr int kMergeThreads = 1024;

// Exclusive prefix sum over the workgroup of one value per thread; also
// returns the total.
__device__ __forceinline__ int block_exclusive_scan(int v, int* s_scan, int& total)
{
    const int tid = threadIdx.x;
    __syncthreads();
    s_scan[tid] = v;
    __syncthreads();
    for (int off = 1; off < kMergeThreads; off <<= 1) {
        const int x = tid >= off ? s_scan[tid - off] : 0;
        __syncthreads();
        s_scan[tid] += x;
        __syncthreads();
    }
    total = s_scan[kMergeThreads - 1];
    return s_scan[tid] - v;
}

// Spikes of one neuron (sorted times ts[0 .. c)) whose float bits are <= x.
__device__ __forceinline__ int count_le(const float* __restrict__ ts, int c, uint32_t x)
{
    int lo = 0, hi = c;                    // first index with bits > x
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (__float_as_uint(ts[mid]) <= x) lo = mid + 1; else hi = mid;
    }
    return lo;
}

__global__ __launch_bounds__(kMergeThreads) void k_merge(const float* __restrict__ out_t,
                                                         const int32_t* __restrict__ out_n, int N, int s_max,
                                                         float* __restrict__ ev_t2, int32_t* __restrict__ ev_src2,
                                                         int32_t* __restrict__ ev_n2, int32_t* __restrict__ perm,
                                                         int E2_max, int cap, int32_t* __restrict__ status)
{
    extern __shared__ unsigned long long keys[];   // cap entries (power of two)
    __shared__ int s_scan[kMergeThreads];
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    const int32_t* cnt = out_n + (size_t)b * N;
    const float* tb = out_t + (size_t)b * N * s_max;
    // each thread owns a contiguous run of neurons
    const int per = (N + kMergeThreads - 1) / kMergeThreads;
    const int i0 = min(tid * per, N), i1 = min(i0 + per, N);
    int local = 0;
    for (int i = i0; i < i1; ++i) local += min(max(cnt[i], 0), s_max);
    int total = 0;
    int pos = block_exclusive_scan(local, s_scan, total);
    const int kept = min(total, E2_max);
    // keys sorted: every spike when they fit, else the kept earliest
    const int held = total <= cap ? total : kept;
    int n2 = 2;
    while (n2 < held) n2 <<= 1;
    for (int e = tid; e < n2; e += kMergeThreads) keys[e] = ~0ull;
    __syncthreads();
    if (total <= cap) {
        // every spike fits: gather all of them
        for (int i = i0; i < i1; ++i) {
            const int c = min(max(cnt[i], 0), s_max);
            const float* ts = tb + (size_t)i * s_max;
            for (int s = 0; s < c; ++s, ++pos)
                keys[pos] = ((unsigned long long)__float_as_uint(ts[s]) << 32) | (unsigned int)(i * s_max + s);
        }
    } else {
        // the smallest float bits x with at least `kept` spikes at or before x
        uint32_t lo = 0u, hi = 0x7f800000u;             // +inf bits: every spike
        while (lo < hi) {
            const uint32_t mid = lo + ((hi - lo) >> 1);
            int le = 0;
            for (int i = i0; i < i1; ++i) le += count_le(tb + (size_t)i * s_max, min(max(cnt[i], 0), s_max), mid);
            int all = 0;
            (void)block_exclusive_scan(le, s_scan, all);
            if (all >= kept) hi = mid; else lo = mid + 1;
        }
        const uint32_t xk = lo;
        // spikes before xk, then the ones at xk in neuron order, up to kept
        int nlt = 0, neq = 0;
        for (int i = i0; i < i1; ++i) {
            const float* ts = tb + (size_t)i * s_max;
            const int c = min(max(cnt[i], 0), s_max);
            const int lt = xk > 0u ? count_le(ts, c, xk - 1u) : 0;
            nlt += lt;
            neq += count_le(ts, c, xk) - lt;
        }
        int tot_lt = 0, tot_eq = 0;
        int plt = block_exclusive_scan(nlt, s_scan, tot_lt);
        int peq = tot_lt + block_exclusive_scan(neq, s_scan, tot_eq);
        for (int i = i0; i < i1; ++i) {
            const float* ts = tb + (size_t)i * s_max;
            const int c = min(max(cnt[i], 0), s_max);
            for (int s = 0; s < c; ++s) {
                const uint32_t tbits = __float_as_uint(ts[s]);
                const unsigned long long key = ((unsigned long long)tbits << 32) | (unsigned int)(i * s_max + s);
                // (the bounds keep malformed, unsorted lists inside the sort)
                if (tbits < xk) {
                    if (plt < kept) keys[plt] = key;
                    ++plt;
                } else if (tbits == xk) {
                    if (peq < kept) keys[peq] = key;
                    ++peq;
                } else {
                    break;
                }
            }
        }
    }
    __syncthreads();
    // Bitonic sort of the n2 keys.
    for (int size = 2; size <= n2; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int e = tid; e < n2; e += kMergeThreads) {
                int partner = e ^ stride;
                if (partner > e) {
                    bool up = (e & size) == 0;
                    unsigned long long a = keys[e], c = keys[partner];
                    if ((a > c) == up) { keys[e] = c; keys[partner] = a; }
                }
            }
            __syncthreads();
        }
    }
    for (int e = tid; e < E2_max; e += kMergeThreads) {
        size_t o = (size_t)b * E2_max + e;
        if (e < kept) {
            unsigned long long k = keys[e];
            unsigned int lo = (unsigned int)(k & 0xffffffffull);
            ev_t2[o] = __uint_as_float((unsigned int)(k >> 32));
            ev_src2[o] = (int)(lo / (unsigned)s_max);
            if (perm) perm[o] = (int)lo;
        } else {
            ev_t2[o] = INFINITY;
            ev_src2[o] = 0;
            if (perm) perm[o] = -1;
        }
    }
    if (tid == 0) {
        ev_n2[b] = kept;
        if (total > E2_max) atomicOr(&status[LIF_ST_FLAGS], LIF_WARN_MERGE_FULL);
    }
}

__global__ void k_zero_status(int32_t* __restrict__ status)
{
    if (threadIdx.x < LIF_STATUS_WORDS) status[threadIdx.x] = 0;
}

// First-spike readout loss, one workgroup: per sample, logits -t_c / tau0,
// log-softmax, cross-entropy against the label, gradient
// dL/dt_c = -(softmax_c - [c == y]) / (tau0 B) on neurons that fired.
__global__ __launch_bounds__(256) void k_first_spike_ce(const float* __restrict__ out_t,
                                                        const int32_t* __restrict__ out_n, int B, int N, int s_max,
                                                        const int32_t* __restrict__ labels, double tau0,
                                                        double t_silent, float* __restrict__ loss,
                                                        float* __restrict__ grad)
{
    __shared__ double red[256];
    int tid = threadIdx.x;
    size_t tot = (size_t)B * N * s_max;
    for (size_t j = tid; j < tot; j += blockDim.x) grad[j] = 0.0f;
    __syncthreads();
    double acc = 0.0;
    for (int b = tid; b < B; b += blockDim.x) {
        const int32_t* cn = out_n + (size_t)b * N;
        double zmax = -INFINITY;
        for (int c = 0; c < N; ++c) {
            double t = cn[c] > 0 ? (double)out_t[((size_t)b * N + c) * s_max] : t_silent;
            zmax = fmax(zmax, -t / tau0);
        }
        double se = 0.0;
        for (int c = 0; c < N; ++c) {
            double t = cn[c] > 0 ? (double)out_t[((size_t)b * N + c) * s_max] : t_silent;
            se += exp(-t / tau0 - zmax);
        }
        int y = min(max(labels[b], 0), N - 1);
        double ty = cn[y] > 0 ? (double)out_t[((size_t)b * N + y) * s_max] : t_silent;
        acc += -(-ty / tau0 - zmax - log(se));
        for (int c = 0; c < N; ++c) {
            if (cn[c] <= 0) continue;
            double t = (double)out_t[((size_t)b * N + c) * s_max];
            double pz = exp(-t / tau0 - zmax) / se;
            double gz = (pz - (c == y ? 1.0 : 0.0)) / (double)B;
            grad[((size_t)b * N + c) * s_max] = (float)(-gz / tau0);
        }
    }
    red[tid] = acc;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
        if (tid < off) red[tid] += red[tid + off];
        __syncthreads();
    }
    if (tid == 0) loss[0] = (float)(red[0] / (double)B);
}

}  // namespace lif

extern "C" size_t lif_merge_workspace_size(int B, int N, int s_max, int E2_max)
{
    (void)B; (void)N; (void)s_max; (void)E2_max;
    return 256;
}

extern "C" int lif_merge_spikes(const float* out_t, const int32_t* out_n, int B, int N, int s_max, float* ev_t2,
                                int32_t* ev_src2, int32_t* ev_n2, int32_t* perm, int E2_max, int32_t* status,
                                void* ws, size_t ws_bytes, lif_stream_t stream_)
{
    hipStream_t stream = (hipStream_t)stream_;
    if (B < 0 || N < 1 || s_max < 1 || E2_max < 1) return LIF_ERR_ARG;
    if (!out_t || !out_n || !ev_t2 || !ev_src2 || !ev_n2 || !status || !ws) return LIF_ERR_ARG;
    if (ws_bytes < lif_merge_workspace_size(B, N, s_max, E2_max)) return LIF_ERR_WORKSPACE;
    if (E2_max > LIF_MERGE_MAX) return LIF_ERR_SIZE;
    if ((size_t)N * (size_t)s_max >= ((size_t)1 << 31)) return LIF_ERR_SIZE;
    // Sort capacity: the smallest power of two holding every spike that can
    // be kept, bounded by the LDS budget.
    size_t most = (size_t)N * (size_t)s_max;
    int cap = 2;
    while ((size_t)cap < most && cap < LIF_MERGE_MAX) cap <<= 1;
    TIMED_LAUNCH("merge_status", lif::k_zero_status, dim3(1), dim3(64), 0, stream, status);
    if (B == 0) return lif::check_launch();
    size_t shmem = (size_t)cap * sizeof(unsigned long long);
    // the sort's LDS exceeds the default dynamic-LDS limit; the attribute is
    // set on every call (for the current device; no state kept here)
    if (hipFuncSetAttribute((const void*)lif::k_merge, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)(LIF_MERGE_MAX * sizeof(unsigned long long))) != hipSuccess)
        return LIF_ERR_HIP;
    TIMED_LAUNCH("merge", lif::k_merge, dim3(B), dim3(lif::kMergeThreads), shmem, stream, out_t, out_n, N, s_max,
                 ev_t2, ev_src2, ev_n2, perm, E2_max, cap, status);
    return lif::check_launch();
}

extern "C" int lif_first_spike_ce(const float* out_t, const int32_t* out_n, int B, int N, int s_max,
                                  const int32_t* labels, double tau0, double t_silent, float* loss,
                                  float* grad_out_t, lif_stream_t stream)
{
    if (B < 1 || N < 1 || s_max < 1 || !(tau0 > 0.0)) return LIF_ERR_ARG;
    if (!out_t || !out_n || !labels || !loss || !grad_out_t) return LIF_ERR_ARG;
    TIMED_LAUNCH("first_spike_ce", lif::k_first_spike_ce, dim3(1), dim3(256), 0, (hipStream_t)stream, out_t, out_n,
                 B, N, s_max, labels, tau0, t_silent, loss, grad_out_t);
    return lif::check_launch();
}
