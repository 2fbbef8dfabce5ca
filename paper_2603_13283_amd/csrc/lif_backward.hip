// lif_backward.hip -- exact gradients of the LIF layer's spike times
// (Appendix D.3, Eq. ift_vjp, chained through the hard resets).
//
// Writing each reset as the subtraction of (V_th - V_reset) e^{-(t - t_s)/tm}
// (exact, because V is continuous at input events and equals V_th at t_s),
// spike s of a neuron is the root of
//   F_s = sum_{k: t_k < t_s} w_k K(t_s - t_k)
//         - (V_th - V_reset) sum_{s' < s} e^{-(t_s - t_s')/tm} - V_th,
// K(u) = kappa (e^{-u/tm} - e^{-u/ts}).  The implicit function theorem gives
// dt_s = -(dF_s/dt_s)^{-1} dF_s with dF_s/dt_s = dV/dt at the spike
// = (I(t_s) - V_th)/tm (Eq. mem_dyn), floored by the solver regularisation.
// With mu_s the adjoint of constraint F_s,
//   lambda_s = g_s - ((V_th - V_reset)/tm) sum_{s'' > s} mu_s'' e^{-(t_s'' - t_s)/tm}
//   mu_s     = -lambda_s / max(dV/dt(t_s), reg)                  (k_spike_adjoint)
// and every input event k collects, with P^m_k = sum over the spikes s
// that come after event k of mu_s e^{-(t_s - t_k)/tm} and P^s_k the same
// with ts,
//   dL/dw_{i, src_k} += kappa (P^m_k - P^s_k)
//   dL/dt_k          += w_{i, src_k} kappa (P^m_k / tm - P^s_k / ts).
// Spike s comes after event k iff k < out_k[s], the forward pass's own count
// of the events consumed before the spike (not a comparison of float32
// times, which can round a spike onto the time of the event before it; the
// offset t_s - t_k is then taken as 0).
// P^m, P^s obey a reverse recurrence with the same per-event decays as the
// forward scan, P_{k-1} = M P_k + (the spikes with out_k = k),
// which k_event_adjoint walks backwards per (sample, segment, chunk of 64
// neurons that fire), taking only neurons with spikes (the others have no
// gradient): the firing neurons of each sample are listed in neuron order
// first (k_bwd_live).  Each segment starts from the closed-form sums over
// the (few) spikes that follow it, so segments are independent.  The walk
// is staged like the forward walks (decays and times in LDS, weights of the
// next group of events in flight).
//
// Both gradients are bitwise reproducible.  dL/dW sums contributions from
// every sample and segment that see the same (channel, neuron): they are
// added as 64-bit fixed-point integers (integer addition is exact and order
// free) with a power-of-two scale chosen per call so that no sum can
// overflow (k_bwd_scale); dL/dt of an event sums over the neuron tiles,
// chunks, whose partial sums are stored per chunk and added in chunk order.
#include <type_traits>

#include "lif_common.hpp"
#include "lif_host.hpp"
#include "lif_walk.hpp"

namespace lif {

struct BwdLayout {
    int S, E_pad, tiles;
    size_t dec, mu, klast, musum, scale, live, nlive, gw, gt, total;
};

static BwdLayout bwd_layout(int B, int E_max, int C_in, int N, int s_max)
{
    BwdLayout L{};
    L.S = (E_max + kSeg - 1) / kSeg;
    L.E_pad = L.S * kSeg;
    size_t off = 0;
    auto take = [&](size_t bytes) { size_t o = off; off += (bytes + 255) & ~(size_t)255; return o; };
    L.tiles = (N + kWave - 1) / kWave;
    L.dec = take((size_t)B * L.E_pad * sizeof(Decay));
    L.mu = take((size_t)B * N * s_max * sizeof(double));
    L.klast = take((size_t)B * N * sizeof(int32_t));
    L.musum = take((size_t)B * N * sizeof(double));
    L.scale = take(sizeof(double));
    L.live = take((size_t)B * N * sizeof(int32_t));
    L.nlive = take((size_t)B * sizeof(int32_t));
    L.gw = take((size_t)C_in * N * sizeof(long long));
    L.gt = take((size_t)L.tiles * B * E_max * sizeof(double));
    L.total = off + 256;
    return L;
}

// Backward setup in one pass (grid-stride over every thread): the
// fixed-point accumulators of dL/dW set to zero; the decays (A, D) per event,
// dec[B][E_pad], identity past each sample's last event (so that the walks
// stage whole segments); and per (sample, neuron) the reverse recurrence
// over its spikes:
//   lambda_s = g_s - ((V_th - V_reset)/tm) sum_{s'' > s} mu_s'' e^{-(t_s'' - t_s)/tm}
//   mu_s     = -lambda_s / max(dV/dt(t_s), reg)
// with the consumed-event count of its last spike (0 when silent): events
// from there on feed no spike, and sum_s |mu_s|, which bounds the neuron's
// P^m and P^s.
__global__ __launch_bounds__(256) void k_bwd_setup(const float* __restrict__ ev_t, const int32_t* __restrict__ ev_n,
                                                   int B, int E_max, int E_pad, int N, Model m,
                                                   Decay* __restrict__ dec, long long* __restrict__ gw, size_t nW,
                                                   const float* __restrict__ out_t, const int32_t* __restrict__ out_n,
                                                   const float* __restrict__ out_i, const int32_t* __restrict__ out_k,
                                                   const float* __restrict__ grad_out_t, double* __restrict__ mu,
                                                   int32_t* __restrict__ klast, double* __restrict__ musum)
{
    const size_t gtid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t gs = (size_t)gridDim.x * blockDim.x;
    for (size_t i = gtid; i < nW; i += gs) gw[i] = 0;
    const size_t nD = (size_t)B * (size_t)E_pad;
    for (size_t idx = gtid; idx < nD; idx += gs) {
        const int b = (int)(idx / (size_t)E_pad), k = (int)(idx % (size_t)E_pad);
        Decay d{1.0, 1.0, 0.0, 0.0};
        if (k < clamp_count(ev_n[b], E_max)) {
            const float* t = ev_t + (size_t)b * E_max;
            const double dt = (double)t[k] - (k > 0 ? (double)t[k - 1] : 0.0);
            d.A = exp(-dt * m.inv_tm);
            d.D = exp(-dt * m.inv_ts);
        }
        dec[idx] = d;
    }
    const size_t nn = (size_t)B * (size_t)N;
    for (size_t idx = gtid; idx < nn; idx += gs) {
        const int ns = min(out_n[idx], m.s_max);
        const size_t o = idx * (size_t)m.s_max;
        const double ms = spike_adjoints(m, ns, out_t + o, out_i + o, grad_out_t + o, mu + o);
        musum[idx] = ms;
        // a neuron whose spikes all have mu = 0 adds exactly 0 everywhere, so
        // it is not walked (a NaN sum keeps it)
        klast[idx] = ns > 0 && ms != 0.0 ? out_k[o + ns - 1] : 0;
    }
}

// Fixed-point scale of the dL/dW sums (one workgroup): every contribution
// kappa (P^m - P^s) of a neuron is at most 2 kappa sum_s |mu_s| in size and a
// sum takes at most one contribution per event of the batch, so with
// bound = 2 kappa max_neuron(sum_s |mu_s|) (events in the batch) the scale
// 2^(62 - ceil(log2 bound)) keeps every sum below 2^62.
constexpr int kScaleThreads = 1024;

__global__ __launch_bounds__(kScaleThreads) void k_bwd_scale(const double* __restrict__ musum, size_t nn,
                                                             const int32_t* __restrict__ ev_n, int B, int E_max,
                                                             double kappa, double* __restrict__ scale)
{
    __shared__ double s_max[kScaleThreads];
    __shared__ double s_ev[kScaleThreads];
    double mx = 0.0, ev = 0.0;
    for (size_t i = threadIdx.x; i < nn; i += kScaleThreads) mx = fmax(mx, musum[i]);
    for (int b = threadIdx.x; b < B; b += kScaleThreads) ev += (double)clamp_count(ev_n[b], E_max);
    s_max[threadIdx.x] = mx;
    s_ev[threadIdx.x] = ev;
    __syncthreads();
    for (int off = kScaleThreads / 2; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off) {
            s_max[threadIdx.x] = fmax(s_max[threadIdx.x], s_max[threadIdx.x + off]);
            s_ev[threadIdx.x] += s_ev[threadIdx.x + off];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const double bound = 2.0 * kappa * s_max[0] * fmax(s_ev[0], 1.0);
        int ex = 0;
        if (bound > 0.0 && isfinite(bound)) frexp(bound, &ex);    // bound < 2^ex
        scale[0] = ldexp(1.0, 62 - ex);
    }
}

// The neurons of each sample that fire, in neuron order (one workgroup per
// sample: a ballot and a prefix sum over the waves per round of 256).
constexpr int kLiveThreads = 256;

__global__ __launch_bounds__(kLiveThreads) void k_bwd_live(const int32_t* __restrict__ klast, int N,
                                                           int32_t* __restrict__ live, int32_t* __restrict__ nlive)
{
    __shared__ int s_cnt[kLiveThreads / kWave];
    const int b = blockIdx.x, wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    int base = 0;
    for (int n0 = 0; n0 < N; n0 += kLiveThreads) {
        const int n = n0 + (int)threadIdx.x;
        const bool f = n < N && klast[(size_t)b * N + n] > 0;
        const unsigned long long bal = __ballot(f);
        const int below = __popcll(bal & ((1ull << lane) - 1ull));
        if (lane == 0) s_cnt[wave] = __popcll(bal);
        __syncthreads();
        int off = base, tot = 0;
        for (int q = 0; q < kLiveThreads / kWave; ++q) {
            if (q < wave) off += s_cnt[q];
            tot += s_cnt[q];
        }
        if (f) live[(size_t)b * N + off + below] = n;
        base += tot;
        __syncthreads();
    }
    if (threadIdx.x == 0) nlive[b] = base;
}

// Accumulators -> float32 outputs: dL/dW from fixed point, dL/dt as the sum
// of the chunks' partial sums in chunk order (0 on padding).
__global__ __launch_bounds__(256) void k_bwd_convert(const long long* __restrict__ gw, const double* __restrict__ scale,
                                                     float* __restrict__ grad_WT, size_t nW,
                                                     const double* __restrict__ gt,
                                                     const int32_t* __restrict__ nlive,
                                                     const int32_t* __restrict__ ev_n, int E_max,
                                                     float* __restrict__ grad_ev_t, size_t nT)
{
    const size_t gtid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t gs = (size_t)gridDim.x * blockDim.x;
    const double inv = 1.0 / scale[0];
    for (size_t i = gtid; i < nW; i += gs) grad_WT[i] = (float)((double)gw[i] * inv);
    if (gt)
        for (size_t i = gtid; i < nT; i += gs) {
            const int b = (int)(i / (size_t)E_max), k = (int)(i % (size_t)E_max);
            double s = 0.0;
            if (k < clamp_count(ev_n[b], E_max)) {
                const int chunks = (nlive[b] + kWave - 1) / kWave;
                for (int q = 0; q < chunks; ++q) s += gt[(size_t)q * nT + i];
            }
            grad_ev_t[i] = (float)s;
        }
}

// One wave per (sample, segment, chunk of 64 firing neurons), walking the
// segment's events backwards: at event k, dL/dw += kappa (P^m - P^s) (one
// fixed-point integer atomic per live lane) and the chunk's part of dL/dt_k,
// the sum over lanes of w kappa (P^m/tm - P^s/ts), is stored; then P decays
// to event k-1 and takes the spikes with out_k = k (those between events
// k-1 and k).  A lane is live while its neuron has a spike after the event.
constexpr int kSpkBatch = 8;
constexpr int kPre = 4;

__global__ __launch_bounds__(kWave * kWalkWaves) void k_event_adjoint(
    const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src, const int32_t* __restrict__ ev_n, int E_max,
    int E_pad, const float* __restrict__ WT, int C_in, int N, int tiles, int S, int items, Model m,
    const Decay* __restrict__ dec, const float* __restrict__ out_t, const int32_t* __restrict__ out_n,
    const int32_t* __restrict__ out_k, const double* __restrict__ mu, const int32_t* __restrict__ klast,
    const int32_t* __restrict__ live_list, const int32_t* __restrict__ nlive, const double* __restrict__ scale_p,
    long long* __restrict__ gWT, double* __restrict__ gT, size_t nT)
{
    __shared__ double2 s_ad[kWalkWaves][kSeg];
    __shared__ float s_t[kWalkWaves][kSeg];
    WalkCoords c;
    if (!walk_coords<1>(items, tiles, S, ev_n, E_max, N, c)) return;
    // the lane's neuron: entry tile * 64 + lane of the sample's list of
    // firing neurons (chunks past the list have nothing to do)
    const int nl = nlive[c.b];
    if (c.tile * kWave >= nl) return;
    const int lane = c.lane;
    const int wv = (int)threadIdx.x / kWave;
    c.live = c.tile * kWave + lane < nl;
    c.n0 = c.live ? live_list[(size_t)c.b * N + c.tile * kWave + lane] : 0;
    const int n = c.n0;
    const float* tt = ev_t + (size_t)c.b * E_max;
    const int kl = c.live ? klast[(size_t)c.b * N + n] : 0;
    const int ns = c.live ? min(out_n[(size_t)c.b * N + n], m.s_max) : 0;
    const bool liv = kl > c.k0;
    // this chunk's part of dL/dt of the segment's events
    double* gt = gT ? gT + (size_t)c.tile * nT + (size_t)c.b * E_max + c.k0 : nullptr;
    if (__ballot(liv) == 0ull) {
        if (gt && lane < c.cnt) gt[lane] = 0.0;
        return;
    }
    const double scale = scale_p[0];
    double2* lad = s_ad[wv];
    float* lt = s_t[wv];
    const Stage st = stage_segment(c, ev_src + (size_t)c.b * E_max + c.k0, dec + (size_t)c.b * E_pad + c.k0, WT,
                                   C_in, N, lad, nullptr, nullptr);
#pragma unroll
    for (int h = 0; h < kSrcRegs; ++h) {
        const int e = h * kWave + lane;
        if (e < c.cnt) lt[e] = tt[c.k0 + e];
    }
    wave_lds_sync();
    const int elast = c.k0 + c.cnt - 1;
    const double tk = (double)lt[c.cnt - 1];
    const size_t base = ((size_t)c.b * N + n) * (size_t)m.s_max;
    const float* ts = out_t + base;
    const int32_t* ks = out_k + base;
    const double* mo = mu + base;
    // One pass over the lane's spikes (from the first one past the
    // segment's start, found by bisection when the list is long), in
    // batches of kSpkBatch loaded together: the closed-form P at the
    // segment's last event from the spikes after it, and the last kPre
    // spikes inside the segment (pk[0] the latest).
    int q0 = 0;
    if (__ballot(liv && ns > 2 * kSpkBatch)) {
        int hi = liv ? ns : 0;
        while (q0 < hi) {
            const int mid = (q0 + hi) >> 1;
            if (ks[mid] > c.k0) hi = mid; else q0 = mid + 1;
        }
    }
    double Pm = 0.0, Ps = 0.0;
    int pk[kPre];
    float pt[kPre];
    double pm[kPre];
#pragma unroll
    for (int u = 0; u < kPre; ++u) {
        pk[u] = -1;
        pt[u] = 0.0f;
        pm[u] = 0.0;
    }
    int nin = 0, sp = q0;                        // spikes inside the segment; first spike after it
    for (int qb = q0; __ballot(liv && qb < ns); qb += kSpkBatch) {
        int kq[kSpkBatch];
        float tq[kSpkBatch];
        double mq[kSpkBatch];
#pragma unroll
        for (int u = 0; u < kSpkBatch; ++u) {
            const int q = min(qb + u, max(ns - 1, 0));
            kq[u] = ks[q];
            tq[u] = ts[q];
            mq[u] = mo[q];
        }
#pragma unroll
        for (int u = 0; u < kSpkBatch; ++u) {
            if (!liv || qb + u >= ns) continue;
            if (kq[u] > elast) {
                const double du = fmax((double)tq[u] - tk, 0.0);
                Pm += mq[u] * exp(-du * m.inv_tm);
                Ps += mq[u] * exp(-du * m.inv_ts);
            } else {
                sp = qb + u + 1;
                if (kq[u] > c.k0) {
#pragma unroll
                    for (int v = kPre - 1; v > 0; --v) {
                        pk[v] = pk[v - 1];
                        pt[v] = pt[v - 1];
                        pm[v] = pm[v - 1];
                    }
                    pk[0] = kq[u];
                    pt[0] = tq[u];
                    pm[0] = mq[u];
                    ++nin;
                }
            }
        }
    }
    // A wave where some lane has more than kPre spikes inside the segment (a
    // burst) walks with each further spike loaded when it is reached (those
    // loads then wait behind the atomics); otherwise the walk loads nothing
    // but the weights.
    const bool burst = __ballot(nin > kPre) != 0ull;
    const double kap = m.kappa;
    auto walk = [&](auto burst_tag) {
        constexpr bool kBurst = decltype(burst_tag)::value;
        int taken = 0;                           // spikes of the segment taken so far
        int knext = pk[0];
        double tnext = (double)pt[0], mnext = pm[0];
        auto advance = [&]() {
            ++taken;
#pragma unroll
            for (int u = 0; u + 1 < kPre; ++u) {
                pk[u] = pk[u + 1];
                pt[u] = pt[u + 1];
                pm[u] = pm[u + 1];
            }
            pk[kPre - 1] = -1;
            knext = pk[0];
            tnext = (double)pt[0];
            mnext = pm[0];
            if (kBurst && taken >= kPre) {
                const int q = sp - 1 - taken;
                const bool in = q >= 0 && taken < nin;
                knext = in ? ks[max(q, 0)] : -1;
                tnext = in ? (double)ts[max(q, 0)] : 0.0;
                mnext = in ? mo[max(q, 0)] : 0.0;
            }
        };
        auto group = [&](int g, const float (&w)[kGrp][1]) {
            double ca[kGrp];
            long long ga[kGrp];
            const int oreg = g * kGrp < kWave ? st.off[0] : st.off[kSrcRegs - 1];
#pragma unroll
            for (int jj = kGrp - 1; jj >= 0; --jj) {
                const int e = g * kGrp + jj;
                ca[jj] = 0.0;
                ga[jj] = 0;
                if (e >= c.cnt) continue;
                ga[jj] = liv ? llrint(kap * (Pm - Ps) * scale) : 0;
                if (gt && liv) ca[jj] = (double)w[jj][0] * kap * (Pm * m.inv_tm - Ps * m.inv_ts);
                if (e > 0) {
                    const double2 ad = lad[e];
                    Pm *= ad.x;
                    Ps *= ad.y;
                    const double tp = (double)lt[e - 1];
                    // spikes between events e - 1 and e (out_k = e)
                    while (knext >= c.k0 + e) {
                        const double u = fmax(tnext - tp, 0.0);
                        Pm += mnext * exp(-u * m.inv_tm);
                        Ps += mnext * exp(-u * m.inv_ts);
                        advance();
                    }
                }
            }
            // the group's weight-gradient terms after its walk, so that the
            // waits for the next weights do not wait for the atomics
#pragma unroll
            for (int jj = 0; jj < kGrp; ++jj) {
                const int e = g * kGrp + jj;
                const int roff = __builtin_amdgcn_readlane(oreg, e & (kWave - 1));
                if (ga[jj] != 0)
                    atomicAdd((unsigned long long*)&gWT[(size_t)(roff >> 2) + (size_t)n],
                              (unsigned long long)ga[jj]);
            }
            if (gt) {
                const double r = group_sum8(ca, lane);
                const int j = ((lane >> 5) & 1) * 4 + ((lane >> 4) & 1) * 2 + ((lane >> 3) & 1);
                const int e = g * kGrp + j;
                if ((lane & 7) == 0 && e < c.cnt) gt[e] = r;
            }
        };
        // groups from the last backwards, the weights of the next one in flight
        const int ng = (c.cnt + kGrp - 1) / kGrp;
        float wa[kGrp][1], wb[kGrp][1];
        load_grp<1>(st, (ng - 1) * kGrp, wa);
        for (int g = ng - 1; g >= 0; g -= 2) {
            if (g >= 1) load_grp<1>(st, (g - 1) * kGrp, wb);
            group(g, wa);
            if (g < 1) break;
            if (g >= 2) load_grp<1>(st, (g - 2) * kGrp, wa);
            group(g - 1, wb);
        }
    };
    if (burst) walk(std::true_type{});
    else walk(std::false_type{});
}

int backward_impl(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max, const float* WT,
                  int C_in, int N, const lif_params* p, const float* out_t, const int32_t* out_n,
                  const float* out_i, const int32_t* out_k, const float* grad_out_t, float* grad_WT,
                  float* grad_ev_t, void* ws, size_t ws_bytes, hipStream_t stream)
{
    int rc = check_params(p);
    if (rc) return rc;
    if (B < 0 || E_max < 0 || C_in < 1 || N < 1) return LIF_ERR_ARG;
    if (!WT || !out_t || !out_n || !out_i || !out_k || !grad_out_t || !grad_WT || !ws) return LIF_ERR_ARG;
    if (B > 0 && !ev_n) return LIF_ERR_ARG;
    if ((size_t)B * (size_t)E_max > 0 && (!ev_t || !ev_src)) return LIF_ERR_ARG;
    if ((size_t)C_in * (size_t)N >= ((size_t)1 << 29)) return LIF_ERR_SIZE;   // 32-bit W^T byte offsets
    BwdLayout L = bwd_layout(B, E_max, C_in, N, p->s_max);
    if (ws_bytes < L.total) return LIF_ERR_WORKSPACE;
    Model m = make_model(*p);
    char* base = (char*)(((uintptr_t)ws + 255) & ~(uintptr_t)255);
    Decay* dec = (Decay*)(base + L.dec);
    double* mu = (double*)(base + L.mu);
    int32_t* klast = (int32_t*)(base + L.klast);
    int32_t* live = (int32_t*)(base + L.live);
    int32_t* nlive = (int32_t*)(base + L.nlive);
    double* musum = (double*)(base + L.musum);
    double* scale = (double*)(base + L.scale);
    long long* gw = (long long*)(base + L.gw);
    double* gt = grad_ev_t ? (double*)(base + L.gt) : nullptr;
    size_t nW = (size_t)C_in * N, nT = (size_t)B * E_max, nn = (size_t)B * N;
    const size_t nD = (size_t)B * L.E_pad;
    {
        size_t work = nW;
        if (nD > work) work = nD;
        if (nn > work) work = nn;
        size_t blocks = (work + 255) / 256;
        if (blocks > 2048) blocks = 2048;
        if (blocks < 1) blocks = 1;
        TIMED_LAUNCH("bwd_setup", k_bwd_setup, dim3((unsigned)blocks), dim3(256), 0, stream, ev_t, ev_n, B, E_max,
                     L.E_pad, N, m, dec, gw, nW, out_t, out_n, out_i, out_k, grad_out_t, mu, klast, musum);
    }
    TIMED_LAUNCH("bwd_scale", k_bwd_scale, dim3(1), dim3(kScaleThreads), 0, stream, musum, nn, ev_n, B, E_max,
                 m.kappa, scale);
    if (B > 0) TIMED_LAUNCH("bwd_live", k_bwd_live, dim3((unsigned)B), dim3(kLiveThreads), 0, stream, klast, N, live, nlive);
    const int tiles = (N + kWave - 1) / kWave;
    const size_t items = (size_t)B * L.S * tiles;
    if (items > 0x7fffffff) return LIF_ERR_SIZE;
    const unsigned blocks = (unsigned)((items + kWalkWaves - 1) / kWalkWaves);
    if (items) TIMED_LAUNCH("event_adjoint", k_event_adjoint, dim3(blocks), dim3(kWave * kWalkWaves), 0, stream,
                            ev_t, ev_src, ev_n, E_max, L.E_pad, WT, C_in, N, tiles, L.S, (int)items, m, dec, out_t,
                            out_n, out_k, mu, klast, live, nlive, scale, gw, gt, nT);
    TIMED_LAUNCH("bwd_convert", k_bwd_convert, dim3(1024), dim3(256), 0, stream, gw, scale, grad_WT, nW, gt, nlive,
                 ev_n, E_max, grad_ev_t, nT);
    return check_launch();
}

}  // namespace lif

extern "C" size_t lif_layer_backward_workspace_size(int B, int E_max, int C_in, int N_out, const lif_params* p)
{
    if (B < 0 || E_max < 0 || C_in < 1 || N_out < 1 || !p || p->s_max < 1) return 0;
    return lif::bwd_layout(B, E_max, C_in, N_out, p->s_max).total;
}

extern "C" int lif_layer_backward(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                                  const float* WT, int C_in, int N_out, const lif_params* p, const float* out_t,
                                  const int32_t* out_n, const float* out_i, const int32_t* out_k,
                                  const float* grad_out_t, float* grad_WT, float* grad_ev_t, void* ws,
                                  size_t ws_bytes, lif_stream_t stream)
{
    return lif::backward_impl(ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, p, out_t, out_n, out_i, out_k,
                              grad_out_t, grad_WT, grad_ev_t, ws, ws_bytes, (hipStream_t)stream);
}
