// lif_chunked.hip -- the paper's own chunked scheme (Sec. 3.2.1 "Speculative
// execution" and "Fixed compute budget", Appendix E.2), for studies of the
// chunk size and of the work retained (Appendix G).
//
// One wave per (sample, neuron).  Each iteration takes the next K = 64 M
// input events of the neuron's queue (lane l holds events l M .. l M + M - 1
// of the chunk) and:
//   * composes each lane's affine maps in the eigen-coordinates (U, J) and
//     takes an exclusive scan of the lane maps across the wave, so every
//     lane knows the state entering its events;
//   * tests every interval closed by one of its events with the interval
//     rule of Sec. 3.2.2 (V at the interval's end, or at the stationary
//     point of Eq. t_vmax when it lies inside, reaching V_th);
//   * commits the first crossing only: its spike time is bracketed as in
//     Appendix D.2 and found by multisection (each round the 64 lanes test
//     64 points of the bracket; the bracket shrinks 64-fold per round, until
//     its ends are adjacent doubles), V is hard-reset, and the next
//     iteration starts from the spike with the same pending event (the
//     chunk's later events were processed and are discarded);
//   * without a crossing consumes all its events; the chunk that holds the
//     last event also tests the interval after it, up to t_end.
// At most C iterations run per neuron and at most s_max spikes are kept; the
// neuron's consumed and processed event counts give the work retention.
// The same walk takes the per-neuron queues of a layer with synaptic delays
// (QUEUE: neuron i's arrival times and the sample's event index of each
// entry, built by lif_delay_queues); out_k then counts events of the
// neuron's own queue.
#include "lif_common.hpp"
#include "lif_scan.hpp"
#include "lif_host.hpp"

namespace lif {

constexpr int kChunkWaves = 4;
constexpr int kChunkLdsC = 2048;        // weight-column entries staged in LDS per wave (8 KB)

// V of the no-reset trajectory u after a state (V0, I0) (Eq. mem_pot).
__device__ __forceinline__ double v_after(const Model& m, double V0, double I0, double u)
{
    const double em = exp(-u * m.inv_tm), es = exp(-u * m.inv_ts);
    return V0 * em + m.kappa * I0 * (em - es);
}

// The interval rule (Sec. 3.2.2) on an interval of length L > 0 from
// (V0, I0), A = e^{-L/tm}, D = e^{-L/ts}: crossing when V(L) >= V_th or when
// the stationary point of Eq. t_vmax lies inside with V >= V_th there; hi is
// the end of the root bracket (the stationary point when it lies inside,
// else L).  Intervals that fail the no-crossing screen of screen_value
// (V0 + max(I0 - V_th, 0) L / tm below the threshold) are rejected first:
// they cannot cross, so the rule's outcome is unchanged.
__device__ __forceinline__ bool interval_rule(const Model& m, double V0, double I0, double L, double A, double D,
                                              double& hi)
{
    hi = L;
    if (V0 + fmax(I0 - m.th, 0.0) * (L * m.inv_tm) < m.th_lo) return false;
    const double vend = V0 * A + m.kappa * I0 * (A - D);
    const double Dm = V0 * (m.tm - m.ts) + I0 * m.ts;
    const bool has_max = I0 > V0 && Dm > 0.0;
    double tv = INFINITY;
    if (has_max) tv = m.c_tv * log(I0 * m.tm / Dm);
    const bool inside = has_max && tv < L;
    hi = inside ? tv : L;
    return vend >= m.th || (inside && v_after(m, V0, I0, tv) >= m.th);
}

// Smallest double u in (0, hi] with V(u) >= V_th (V(hi) >= V_th, V rising on
// [0, hi]): 64-way multisection, wave-uniform result.
__device__ double spike_offset(const Model& m, double V0, double I0, double hi)
{
    const int lane = (int)threadIdx.x % kWave;
    double lo = 0.0;
    for (int round = 0; round < 64; ++round) {
        if (!(nextafter(lo, INFINITY) < hi)) break;
        const double x = lane == kWave - 1 ? hi : lo + (hi - lo) * ((double)(lane + 1) / (double)kWave);
        const bool ok = lane == kWave - 1 || v_after(m, V0, I0, x) >= m.th;
        const unsigned long long bal = __ballot(ok);
        const int f = __ffsll((long long)bal) - 1;
        const double nh = __shfl(x, f, kWave);
        const double nl = f > 0 ? __shfl(x, f - 1, kWave) : lo;
        if (nh == hi && nl == lo) break;
        hi = nh;
        lo = fmax(lo, nl);
    }
    return hi;
}

struct LaneMap {
    double aU, bU, aJ, bJ;   // U_out = aU U_in + bU, J_out = aJ J_in + bJ
};

template <int M, bool QUEUE>
__global__ __launch_bounds__(kWave * kChunkWaves) void k_chunked(
    const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src, const int32_t* __restrict__ ev_n,
    const int32_t* __restrict__ q_k, int B, int E_max, const float* __restrict__ WT, int C_in, int N, Model m,
    int C_budget, float* __restrict__ out_t,
    int32_t* __restrict__ out_n, float* __restrict__ out_i, int32_t* __restrict__ out_k,
    int32_t* __restrict__ consumed, int32_t* __restrict__ processed, int32_t* __restrict__ status)
{
    constexpr int K = kWave * M;
    __shared__ float s_w[kChunkWaves][kChunkLdsC];
    const int lane = (int)threadIdx.x % kWave, wave = (int)threadIdx.x / kWave;
    // waves in neuron-major order: the waves of a workgroup mostly share a
    // neuron, so their loads of its weight column hit the same lines
    const size_t item = (size_t)blockIdx.x * kChunkWaves + wave;
    if (item >= (size_t)B * N) return;
    const int n = (int)(item / (size_t)B), b = (int)(item % (size_t)B);
    const size_t idx = (size_t)b * N + n;
    const int nb = clamp_count(ev_n[b], E_max);
    // the neuron's queue: the sample's events, or (QUEUE) its own arrivals
    const float* tt = ev_t + (QUEUE ? idx : (size_t)b) * (size_t)E_max;
    const int32_t* src = ev_src + (size_t)b * E_max;
    const int32_t* qk = QUEUE ? q_k + idx * (size_t)E_max : nullptr;
    float* st = out_t + idx * (size_t)m.s_max;
    float* si = out_i ? out_i + idx * (size_t)m.s_max : nullptr;
    int32_t* sk = out_k ? out_k + idx * (size_t)m.s_max : nullptr;
    // the neuron's weight column W^T[:, n] in the wave's LDS slice (lanes of
    // one event chunk read random rows of it); from global memory when it
    // does not fit.  Each wave writes and reads only its own slice, and LDS
    // operations of one wave complete in order.
    const bool lds_w = C_in <= kChunkLdsC;
    if (lds_w) {
        for (int c = lane; c < C_in; c += kWave) s_w[wave][c] = WT[(size_t)c * N + n];
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    double t_cur = 0.0, V = 0.0, I = 0.0;
    int k = 0, chunks = 0, ns = 0;
    long long work = 0;
    bool finished = false;
    while (!finished && ns < m.s_max && chunks < C_budget) {
        ++chunks;
        const int end = min(k + K, nb);
        work += end - k;
        // the lane's events: times, weights, and each interval's decays
        double te[M], L[M], A[M], D[M];
        float w[M];
        bool valid[M];
#pragma unroll
        for (int j = 0; j < M; ++j) {
            const int e = k + lane * M + j;
            valid[j] = e < end;
            te[j] = valid[j] ? (double)tt[e] : 0.0;
            const int se = QUEUE ? min(max(valid[j] ? qk[e] : 0, 0), max(nb - 1, 0)) : e;
            const int c = valid[j] ? clamp_src(src[se], C_in) : 0;
            w[j] = valid[j] ? (lds_w ? s_w[wave][c] : WT[(size_t)c * N + n]) : 0.0f;
        }
        // the time before each event: the previous event's, t_cur for the
        // chunk's first
        const double prev_last = wave_shr1(te[M - 1], t_cur);
#pragma unroll
        for (int j = 0; j < M; ++j) {
            const double tp = j > 0 ? te[j - 1] : prev_last;
            L[j] = valid[j] ? te[j] - tp : 0.0;
            A[j] = exp(-L[j] * m.inv_tm);
            D[j] = exp(-L[j] * m.inv_ts);
        }
        // the lane's composed map, then the exclusive scan over lanes
        LaneMap f{1.0, 0.0, 1.0, 0.0};
#pragma unroll
        for (int j = 0; j < M; ++j) {
            if (!valid[j]) continue;
            const double x = (double)w[j];
            f.aU *= A[j];
            f.bU = fma(A[j], f.bU, x);
            f.aJ *= D[j];
            f.bJ = fma(D[j], f.bJ, x);
        }
        LaneMap inc = f;                      // inclusive scan: maps of lanes 0 .. l
        scan_maps_up(inc.aU, inc.bU, lane);
        scan_maps_up(inc.aJ, inc.bJ, lane);
        const LaneMap ex{wave_shr1(inc.aU, 1.0), wave_shr1(inc.bU, 0.0), wave_shr1(inc.aJ, 1.0),
                         wave_shr1(inc.bJ, 0.0)};
        const double U0 = V / m.kappa + I, J0 = I;
        double U = fma(ex.aU, U0, ex.bU), J = fma(ex.aJ, J0, ex.bJ);
        // the lane's intervals in order; the first crossing's data kept
        int jc = -1;
        double cV = 0.0, cI = 0.0, chi = 0.0;
#pragma unroll
        for (int j = 0; j < M; ++j) {
            if (!valid[j]) continue;
            if (jc < 0 && L[j] > 0.0) {
                double hi;
                const double V0 = m.kappa * (U - J), I0 = J;
                if (interval_rule(m, V0, I0, L[j], A[j], D[j], hi)) {
                    jc = j;
                    cV = V0;
                    cI = I0;
                    chi = hi;
                }
            }
            const double x = (double)w[j];
            U = fma(A[j], U, x);
            J = fma(D[j], J, x);
        }
        const unsigned long long cross = __ballot(jc >= 0);
        if (cross) {
            const int lc = __ffsll((long long)cross) - 1;
            const int jj = __shfl(jc, lc, kWave);
            const double V0 = __shfl(cV, lc, kWave), I0 = __shfl(cI, lc, kWave), hi = __shfl(chi, lc, kWave);
            const int ecross = k + lc * M + jj;
            const double tstart = (double)__shfl(te[M - 1], max(lc - 1, 0), kWave);
            double t0 = t_cur;
            // the interval's start: the previous event, or t_cur for the chunk's first
            {
                double tp = 0.0;
#pragma unroll
                for (int j = 0; j < M; ++j)
                    if (j == jj - 1) tp = __shfl(te[j], lc, kWave);
                if (jj > 0) t0 = tp;
                else if (lc > 0) t0 = tstart;
            }
            const double tau = spike_offset(m, V0, I0, hi);
            const double Is = I0 * exp(-tau * m.inv_ts);
            if (lane == 0) {
                st[ns] = (float)(t0 + tau);
                if (si) si[ns] = (float)Is;
                if (sk) sk[ns] = ecross;
            }
            ++ns;
            V = m.vr;
            I = Is;
            t_cur = t0 + tau;
            k = ecross;
            continue;
        }
        // no crossing: the chunk's events are consumed
        if (end > k) {
            const int ll = (end - 1 - k) / M;
            const double Ue = __shfl(U, ll, kWave), Je = __shfl(J, ll, kWave);
            // the lane's state after all of its events equals the state after
            // event end - 1 (its later slots are past the chunk)
            V = m.kappa * (Ue - Je);
            I = Je;
            t_cur = (double)tt[end - 1];
        }
        k = end;
        if (end == nb) {
            // the interval after the last event, up to t_end
            const double Lo = m.t_end - t_cur;
            double hi;
            if (Lo > 0.0 && interval_rule(m, V, I, Lo, exp(-Lo * m.inv_tm), exp(-Lo * m.inv_ts), hi)) {
                const double tau = spike_offset(m, V, I, hi);
                const double Is = I * exp(-tau * m.inv_ts);
                if (lane == 0) {
                    st[ns] = (float)(t_cur + tau);
                    if (si) si[ns] = (float)Is;
                    if (sk) sk[ns] = nb;
                }
                ++ns;
                V = m.vr;
                I = Is;
                t_cur = t_cur + tau;
            } else {
                finished = true;
            }
        }
    }
    // padding, counts, work counters, status
    for (int q = ns + lane; q < m.s_max; q += kWave) {
        st[q] = INFINITY;
        if (si) si[q] = 0.0f;
        if (sk) sk[q] = 0;
    }
    if (lane == 0) {
        out_n[idx] = ns;
        if (consumed) consumed[idx] = k;
        if (processed) processed[idx] = (int32_t)min(work, 0x7fffffffll);
        if (ns) {
            atomicAdd(&status[LIF_ST_SPIKES], ns);
            atomicAdd(&status[LIF_ST_ROOT_SOLVES], ns);
        }
        if (ns >= m.s_max) {
            atomicAdd(&status[LIF_ST_CAPPED], 1);
            atomicOr(&status[LIF_ST_FLAGS], LIF_WARN_SPIKE_CAP);
        }
        atomicAdd(&status[LIF_ST_CAND_BLOCKS], chunks);
        atomicAdd(&status[LIF_ST_WALKED_BLOCKS], (int32_t)min(work, 0x7fffffffll));
        if (n == 0) atomicAdd(&status[LIF_ST_EVENTS], nb);
    }
}

__global__ void k_chunked_status_reset(int32_t* __restrict__ status)
{
    if (threadIdx.x < LIF_STATUS_WORDS) status[threadIdx.x] = 0;
}

int launch_chunked_walk(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, const int32_t* q_k, int B,
                        int E_max, const float* WT, int C_in, int N, const Model& m, int K, int C, float* out_t,
                        int32_t* out_n, float* out_i, int32_t* out_k, int32_t* consumed, int32_t* processed,
                        int32_t* status, hipStream_t stream)
{
    TIMED_LAUNCH("chunked_reset", k_chunked_status_reset, dim3(1), dim3(kWave), 0, stream, status);
    const size_t waves = (size_t)B * N;
    if (waves) {
        const dim3 grid((unsigned)((waves + kChunkWaves - 1) / kChunkWaves)), block(kWave * kChunkWaves);
#define LIF_CHUNKED(MM, QQ)                                                                                       \
    TIMED_LAUNCH("chunked", (k_chunked<MM, QQ>), grid, block, 0, stream, ev_t, ev_src, ev_n, q_k, B, E_max, WT, \
                 C_in, N, m, C, out_t, out_n, out_i, out_k, consumed, processed, status)
        if (q_k) {
            switch (K) {
            case 64: LIF_CHUNKED(1, true); break;
            case 128: LIF_CHUNKED(2, true); break;
            default: LIF_CHUNKED(4, true); break;
            }
        } else {
            switch (K) {
            case 64: LIF_CHUNKED(1, false); break;
            case 128: LIF_CHUNKED(2, false); break;
            default: LIF_CHUNKED(4, false); break;
            }
        }
#undef LIF_CHUNKED
    }
    return check_launch();
}

}  // namespace lif

extern "C" int lif_layer_forward_chunked(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B,
                                         int E_max, const float* WT, int C_in, int N_out, const lif_params* p,
                                         int K, int C, float* out_t, int32_t* out_n, float* out_i, int32_t* out_k,
                                         int32_t* consumed, int32_t* processed, int32_t* status,
                                         lif_stream_t stream_)
{
    using namespace lif;
    int rc = validate_forward_args(ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, p, out_t, out_n, status);
    if (rc) return rc;
    if (K != 64 && K != 128 && K != 256) return LIF_ERR_ARG;
    if ((size_t)B * (size_t)N_out >= ((size_t)1 << 31)) return LIF_ERR_SIZE;
    if (C <= 0) C = (E_max + K - 1) / K + p->s_max;    // the paper's budget for an input layer (App. E.2)
    return launch_chunked_walk(ev_t, ev_src, ev_n, nullptr, B, E_max, WT, C_in, N_out, make_model(*p), K, C, out_t,
                               out_n, out_i, out_k, consumed, processed, status, (hipStream_t)stream_);
}
