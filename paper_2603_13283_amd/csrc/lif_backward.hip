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
// and every input event k collects, with P^m_k = sum_{t_s > t_k} mu_s
// e^{-(t_s - t_k)/tm} and P^s_k the same with ts,
//   dL/dw_{i, src_k} += kappa (P^m_k - P^s_k)
//   dL/dt_k          += w_{i, src_k} kappa (P^m_k / tm - P^s_k / ts).
// P^m, P^s obey a reverse recurrence with the same per-event decays as the
// forward scan, P_{k-1} = M P_k + (spike injections in (t_{k-1}, t_k]),
// which k_event_adjoint walks backwards per (sample, 64-neuron tile,
// segment); each segment starts from the closed-form sums over the
// (few) spikes that follow it, so segments are independent.
#include "lif_common.hpp"
#include "lif_host.hpp"

namespace lif {

struct BwdLayout {
    int S;
    size_t dec, mu, last, gw, gt, total;
};

static BwdLayout bwd_layout(int B, int E_max, int C_in, int N, int s_max)
{
    BwdLayout L{};
    L.S = (E_max + kSeg - 1) / kSeg;
    size_t off = 0;
    auto take = [&](size_t bytes) { size_t o = off; off += (bytes + 255) & ~(size_t)255; return o; };
    L.dec = take((size_t)B * E_max * sizeof(Decay));
    L.mu = take((size_t)B * N * s_max * sizeof(double));
    L.last = take((size_t)B * N * sizeof(float));
    L.gw = take((size_t)C_in * N * sizeof(double));
    L.gt = take((size_t)B * E_max * sizeof(double));
    L.total = off + 256;
    return L;
}

__global__ __launch_bounds__(256) void k_bwd_decay(const float* __restrict__ ev_t, const int32_t* __restrict__ ev_n,
                                                   int B, int E_max, Model m, Decay* __restrict__ dec)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (size_t)B * (size_t)E_max) return;
    int b = (int)(idx / (size_t)E_max), k = (int)(idx % (size_t)E_max);
    if (k >= clamp_count(ev_n[b], E_max)) return;
    const float* t = ev_t + (size_t)b * E_max;
    double dt = (double)t[k] - (k > 0 ? (double)t[k - 1] : 0.0);
    Decay d;
    d.A = exp(-dt * m.inv_tm);
    d.D = exp(-dt * m.inv_ts);
    d.C = 0.0;
    d.lk = 0.0;
    dec[idx] = d;
}

__global__ __launch_bounds__(256) void k_fill_zero(double* __restrict__ a, size_t n)
{
    size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    size_t stride = (size_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) a[i] = 0.0;
}

// float64 accumulators -> float32 outputs.
__global__ __launch_bounds__(256) void k_to_float(const double* __restrict__ a, float* __restrict__ out, size_t n)
{
    size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    size_t stride = (size_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) out[i] = (float)a[i];
}

// Per (sample, neuron): reverse recurrence over its spikes.
__global__ __launch_bounds__(256) void k_spike_adjoint(int B, int N, Model m, const float* __restrict__ out_t,
                                                       const int32_t* __restrict__ out_n,
                                                       const float* __restrict__ out_i,
                                                       const float* __restrict__ grad_out_t,
                                                       double* __restrict__ mu, float* __restrict__ last)
{
    size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (size_t)B * (size_t)N) return;
    int ns = min(out_n[idx], m.s_max);
    const float* ts = out_t + idx * (size_t)m.s_max;
    const float* is = out_i + idx * (size_t)m.s_max;
    const float* g = grad_out_t + idx * (size_t)m.s_max;
    double* mo = mu + idx * (size_t)m.s_max;
    double Q = 0.0, mu_next = 0.0;
    double jump = (m.th - m.vr) * m.inv_tm;
    for (int s = ns - 1; s >= 0; --s) {
        if (s + 1 < ns) Q = (Q + mu_next) * exp(-((double)ts[s + 1] - (double)ts[s]) * m.inv_tm);
        double lam = (double)g[s] - jump * Q;
        double vp = fmax(((double)is[s] - m.th) * m.inv_tm, m.reg);
        double mu_s = vp > 0.0 ? -lam / vp : 0.0;
        mo[s] = mu_s;
        mu_next = mu_s;
    }
    last[idx] = ns > 0 ? ts[ns - 1] : -INFINITY;
}

__device__ __forceinline__ double wave_sum(double v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}

__global__ __launch_bounds__(64) void k_event_adjoint(const float* __restrict__ ev_t, const int32_t* __restrict__ ev_src,
                                                      const int32_t* __restrict__ ev_n, int E_max,
                                                      const float* __restrict__ WT, int C_in, int N, int tiles, int S,
                                                      Model m, const Decay* __restrict__ dec,
                                                      const float* __restrict__ out_t,
                                                      const int32_t* __restrict__ out_n,
                                                      const double* __restrict__ mu,
                                                      const float* __restrict__ last, double* __restrict__ gWT,
                                                      double* __restrict__ gT)
{
    int lin = blockIdx.x;
    int tile = lin % tiles;
    int rest = lin / tiles;
    int seg = rest % S;
    int b = rest / S;
    int nb = clamp_count(ev_n[b], E_max);
    int k0 = seg * kSeg;
    if (k0 >= nb) return;
    int k1 = min(k0 + kSeg, nb);
    int n = tile * kWave + (int)threadIdx.x;
    bool act = n < N;
    int nc = min(n, N - 1);
    const float* tt = ev_t + (size_t)b * E_max;
    // Only spikes after the segment's first event matter; skip the wave when
    // no lane has one.
    float tlast = act ? last[(size_t)b * N + nc] : -INFINITY;
    bool live = tlast > tt[k0];
    if (__ballot(live) == 0) return;
    size_t base = ((size_t)b * N + nc) * (size_t)m.s_max;
    const float* ts = out_t + base;
    const double* mo = mu + base;
    int ns = act ? min(out_n[(size_t)b * N + nc], m.s_max) : 0;
    // Closed-form P at the last event of the segment: spikes strictly later.
    double tk = (double)tt[k1 - 1];
    double Pm = 0.0, Ps = 0.0;
    int sp = ns;                 // spikes with index >= sp are later than the current event
    if (live) {
        while (sp > 0 && (double)ts[sp - 1] > tk) --sp;
        for (int s = sp; s < ns; ++s) {
            double u = (double)ts[s] - tk;
            Pm += mo[s] * exp(-u * m.inv_tm);
            Ps += mo[s] * exp(-u * m.inv_ts);
        }
    }
    const int32_t* src = ev_src + (size_t)b * E_max;
    const Decay* d = dec + (size_t)b * E_max;
    for (int k = k1 - 1; k >= k0; --k) {
        int c = clamp_src(src[k], C_in);
        float w = WT[(size_t)c * N + nc];
        double a = m.kappa * (Pm - Ps);
        if (live && a != 0.0) atomicAdd(&gWT[(size_t)c * N + n], a);
        if (gT) {
            double contrib = live ? (double)w * m.kappa * (Pm * m.inv_tm - Ps * m.inv_ts) : 0.0;
            double tot = wave_sum(contrib);
            if (threadIdx.x == 0 && tot != 0.0) atomicAdd(&gT[(size_t)b * E_max + k], tot);
        }
        if (k == k0) break;
        // Step to event k-1: decay over the gap t_k - t_{k-1} and inject the
        // spikes in (t_{k-1}, t_k].
        Decay e = d[k];
        Pm *= e.A;
        Ps *= e.D;
        if (live) {
            double tp = (double)tt[k - 1];
            while (sp > 0 && (double)ts[sp - 1] > tp) {
                --sp;
                double u = (double)ts[sp] - tp;
                Pm += mo[sp] * exp(-u * m.inv_tm);
                Ps += mo[sp] * exp(-u * m.inv_ts);
            }
        }
    }
}

int backward_impl(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max, const float* WT,
                  int C_in, int N, const lif_params* p, const float* out_t, const int32_t* out_n,
                  const float* out_i, const float* grad_out_t, float* grad_WT, float* grad_ev_t, void* ws,
                  size_t ws_bytes, hipStream_t stream)
{
    int rc = check_params(p);
    if (rc) return rc;
    if (B < 0 || E_max < 0 || C_in < 1 || N < 1) return LIF_ERR_ARG;
    if (!WT || !out_t || !out_n || !out_i || !grad_out_t || !grad_WT || !ws) return LIF_ERR_ARG;
    if (B > 0 && !ev_n) return LIF_ERR_ARG;
    if ((size_t)B * (size_t)E_max > 0 && (!ev_t || !ev_src)) return LIF_ERR_ARG;
    BwdLayout L = bwd_layout(B, E_max, C_in, N, p->s_max);
    if (ws_bytes < L.total) return LIF_ERR_WORKSPACE;
    Model m = make_model(*p);
    char* base = (char*)(((uintptr_t)ws + 255) & ~(uintptr_t)255);
    Decay* dec = (Decay*)(base + L.dec);
    double* mu = (double*)(base + L.mu);
    float* last = (float*)(base + L.last);
    double* gw = (double*)(base + L.gw);
    double* gt = grad_ev_t ? (double*)(base + L.gt) : nullptr;
    size_t nW = (size_t)C_in * N, nT = (size_t)B * E_max, nn = (size_t)B * N;
    TIMED_LAUNCH("bwd_zero", k_fill_zero, dim3(1024), dim3(256), 0, stream, gw, nW);
    if (gt && nT) TIMED_LAUNCH("bwd_zero", k_fill_zero, dim3(256), dim3(256), 0, stream, gt, nT);
    if (nT) TIMED_LAUNCH("bwd_decay", k_bwd_decay, dim3((unsigned)((nT + 255) / 256)), dim3(256), 0, stream,
                         ev_t, ev_n, B, E_max, m, dec);
    if (nn) TIMED_LAUNCH("spike_adjoint", k_spike_adjoint, dim3((unsigned)((nn + 255) / 256)), dim3(256), 0,
                         stream, B, N, m, out_t, out_n, out_i, grad_out_t, mu, last);
    int tiles = (N + kWave - 1) / kWave;
    size_t total = (size_t)B * L.S * tiles;
    if (total > 0x7fffffff) return LIF_ERR_SIZE;
    if (total) TIMED_LAUNCH("event_adjoint", k_event_adjoint, dim3((unsigned)total), dim3(kWave), 0, stream,
                            ev_t, ev_src, ev_n, E_max, WT, C_in, N, tiles, L.S, m, dec, out_t, out_n, mu, last, gw,
                            gt);
    TIMED_LAUNCH("bwd_convert", k_to_float, dim3(1024), dim3(256), 0, stream, gw, grad_WT, nW);
    if (gt && nT) TIMED_LAUNCH("bwd_convert", k_to_float, dim3(256), dim3(256), 0, stream, gt, grad_ev_t, nT);
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
                                  const int32_t* out_n, const float* out_i, const float* grad_out_t, float* grad_WT,
                                  float* grad_ev_t, void* ws, size_t ws_bytes, lif_stream_t stream)
{
    return lif::backward_impl(ev_t, ev_src, ev_n, B, E_max, WT, C_in, N_out, p, out_t, out_n, out_i, grad_out_t,
                              grad_WT, grad_ev_t, ws, ws_bytes, (hipStream_t)stream);
}
