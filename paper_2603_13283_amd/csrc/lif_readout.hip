// lif_readout.hip -- the paper's readout and loss (Sec. 3.3, App. C): a
// weighted leaky integrator (LI) per class, with the LIF neuron's V/I
// dynamics and no spikes, fed by the last hidden layer's merged spike queue;
// its logit is the integral of e^{-t/tau_LI} V(t) over [0, tau_max] (Eq.
// weighted_leaky_integrator_full), scaled by a fixed temperature multiplier
// before the softmax cross-entropy.  Also the scatter of queue-time
// gradients back to the spikes that formed the queue (the inverse of the
// layer merge).
//
// The LI state is linear in its inputs and never resets, so the logit is a
// superposition over the queue's events: z_c = sum_e W[src_e, c] G(t_e),
// where G(t0) is the weighted integral of one unit event at t0,
//   G(t0) = kappa e^{-t0/tau_LI} [T_m (1 - e^{-r/T_m}) - T_s (1 - e^{-r/T_s})],
//   r = tau_max - t0, T_x = tau_LI tau_x / (tau_LI + tau_x),
// which is the interval-by-interval closed form of the paper summed over
// intervals.  Every factor is at most 1, so no exponent overflows (the
// product e^{t_i/tau_m} e^{-t_i/T_m} of the printed form is e^{-t_i/tau_LI}).
//
// Passes (no atomics on floating-point values; every sum has a fixed order):
//   k_li_kernel   per event: G and dG/dt0 (lanes are events).
//   k_li_logits   per (sample, 64 classes): lanes are classes, four waves
//                 take contiguous quarters of the queue, W rows gathered per
//                 event; quarters combined in wave order.
//   k_li_ce       per sample: softmax of beta z, the sample's loss and
//                 dL/dz = beta (p - onehot) / B; then the batch mean.
//   k_li_hist     per event: H[b][src] += G (64-bit fixed-point integer
//                 atomics, exact and order-free), so that
//   k_li_grad_w   dL/dW[c][k] = sum_b H[b][c] dL/dz[b][k] (b in order).
//   k_li_grad_t   per event: dL/dt_e = dG(t_e) sum_k W[src_e][k] dL/dz[b][k].
#include "lif_common.hpp"
#include "lif_host.hpp"

namespace lif {

constexpr int kLiThreads = 256;
constexpr double kHistScale = 1099511627776.0;     // 2^40: fixed-point step of H

struct LiModel {
    double kappa, inv_li, Tm, Ts, tau_max, beta;
};

static LiModel make_li(const lif_li_params& q)
{
    LiModel m;
    m.kappa = q.tau_syn / (q.tau_mem - q.tau_syn);
    const bool unweighted = isinf(q.tau_li);
    m.inv_li = unweighted ? 0.0 : 1.0 / q.tau_li;
    m.Tm = unweighted ? q.tau_mem : q.tau_li * q.tau_mem / (q.tau_li + q.tau_mem);
    m.Ts = unweighted ? q.tau_syn : q.tau_li * q.tau_syn / (q.tau_li + q.tau_syn);
    m.tau_max = q.tau_max;
    m.beta = q.beta;
    return m;
}

// G(t0) and dG/dt0 of one unit event (zero at or after tau_max).
__device__ __forceinline__ double2 event_kernel(const LiModel& m, double t0)
{
    if (!(t0 < m.tau_max)) return make_double2(0.0, 0.0);
    const double w0 = exp(-t0 * m.inv_li);
    const double r = m.tau_max - t0;
    const double am = exp(-r / m.Tm), as = exp(-r / m.Ts);
    // T (1 - e^{-r/T}) = -T expm1(-r/T), accurate for small r
    const double G = m.kappa * w0 * (-m.Tm * expm1(-r / m.Tm) + m.Ts * expm1(-r / m.Ts));
    const double dG = -G * m.inv_li + m.kappa * w0 * (as - am);
    return make_double2(G, dG);
}

__global__ __launch_bounds__(kLiThreads) void k_li_kernel(const float* __restrict__ ev_t,
                                                          const int32_t* __restrict__ ev_n, int E_max, LiModel m,
                                                          double2* __restrict__ gk)
{
    const int b = blockIdx.y;
    const int e = blockIdx.x * kLiThreads + threadIdx.x;
    if (e >= E_max) return;
    const int nb = clamp_count(ev_n[b], E_max);
    gk[(size_t)b * E_max + e] = e < nb ? event_kernel(m, (double)ev_t[(size_t)b * E_max + e]) : make_double2(0.0, 0.0);
}

__global__ __launch_bounds__(kLiThreads) void k_li_logits(const int32_t* __restrict__ ev_src,
                                                          const int32_t* __restrict__ ev_n, int E_max,
                                                          const float* __restrict__ WT, int C_in, int ncls,
                                                          const double2* __restrict__ gk, double* __restrict__ z64,
                                                          float* __restrict__ logits)
{
    __shared__ double part[kLiThreads / kWave][kWave];
    const int b = blockIdx.x;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int c = blockIdx.y * kWave + lane;
    const bool live = c < ncls;
    const int nb = clamp_count(ev_n[b], E_max);
    constexpr int nw = kLiThreads / kWave;
    const int per = (nb + nw - 1) / nw;
    const int e0 = min(wave * per, nb), e1 = min(e0 + per, nb);
    const int32_t* src = ev_src + (size_t)b * E_max;
    const double2* g = gk + (size_t)b * E_max;
    double acc = 0.0;
    constexpr int kU = 8;
    for (int e = e0; e < e1; e += kU) {
        float w[kU];
        double G[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int ee = min(e + u, e1 - 1);
            const int s = clamp_src(src[ee], C_in);
            w[u] = live ? WT[(size_t)s * ncls + c] : 0.0f;
            G[u] = e + u < e1 ? g[ee].x : 0.0;
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) acc = fma(G[u], (double)w[u], acc);
    }
    part[wave][lane] = acc;
    __syncthreads();
    if (wave == 0 && live) {
        double z = 0.0;
#pragma unroll
        for (int q = 0; q < nw; ++q) z += part[q][lane];
        z64[(size_t)b * ncls + c] = z;
        if (logits) logits[(size_t)b * ncls + c] = (float)z;
    }
}

// One wave per sample (lanes are classes, ncls <= 64).
__global__ __launch_bounds__(kWave) void k_li_ce(const double* __restrict__ z64, int B, int ncls,
                                                 const int32_t* __restrict__ labels, double beta,
                                                 double* __restrict__ dz, double* __restrict__ loss_b)
{
    const int b = blockIdx.x, c = threadIdx.x;
    const bool live = c < ncls;
    const double y = live ? beta * z64[(size_t)b * ncls + c] : -INFINITY;
    double mx = y;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) mx = fmax(mx, __shfl_xor(mx, off, kWave));
    const double ex = live ? exp(y - mx) : 0.0;
    double sum = ex;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off, kWave);
    const int lab = min(max(labels[b], 0), ncls - 1);
    const double p = ex / sum;
    if (live) dz[(size_t)b * ncls + c] = beta * (p - (c == lab ? 1.0 : 0.0)) / (double)B;
    const double y_lab = __shfl(y, lab, kWave);
    if (c == 0) loss_b[b] = log(sum) - (y_lab - mx);
}

__global__ void k_li_loss(const double* __restrict__ loss_b, int B, float* __restrict__ loss)
{
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    double s = 0.0;
    for (int b = 0; b < B; ++b) s += loss_b[b];
    loss[0] = (float)(s / (double)B);
}

__global__ __launch_bounds__(kLiThreads) void k_fill_u64(unsigned long long* __restrict__ p, size_t n)
{
    const size_t i = (size_t)blockIdx.x * kLiThreads + threadIdx.x;
    if (i < n) p[i] = 0ull;
}

__global__ __launch_bounds__(kLiThreads) void k_li_hist(const int32_t* __restrict__ ev_src,
                                                        const int32_t* __restrict__ ev_n, int E_max, int C_in,
                                                        const double2* __restrict__ gk,
                                                        unsigned long long* __restrict__ H)
{
    const int b = blockIdx.y;
    const int e = blockIdx.x * kLiThreads + threadIdx.x;
    if (e >= clamp_count(ev_n[b], E_max)) return;
    const double G = gk[(size_t)b * E_max + e].x;
    if (G == 0.0) return;
    const long long q = llrint(G * kHistScale);
    atomicAdd(&H[(size_t)b * C_in + clamp_src(ev_src[(size_t)b * E_max + e], C_in)], (unsigned long long)q);
}

__global__ __launch_bounds__(kLiThreads) void k_li_grad_w(const unsigned long long* __restrict__ H, int B, int C_in,
                                                          int ncls, const double* __restrict__ dz,
                                                          float* __restrict__ grad_WT)
{
    const size_t i = (size_t)blockIdx.x * kLiThreads + threadIdx.x;
    if (i >= (size_t)C_in * ncls) return;
    const int c = (int)(i / ncls), k = (int)(i % ncls);
    double s = 0.0;
    for (int b = 0; b < B; ++b) {
        const long long h = (long long)H[(size_t)b * C_in + c];
        if (h) s = fma((double)h / kHistScale, dz[(size_t)b * ncls + k], s);
    }
    grad_WT[i] = (float)s;
}

__global__ __launch_bounds__(kLiThreads) void k_li_grad_t(const int32_t* __restrict__ ev_src,
                                                          const int32_t* __restrict__ ev_n, int E_max,
                                                          const float* __restrict__ WT, int C_in, int ncls,
                                                          const double2* __restrict__ gk,
                                                          const double* __restrict__ dz, float* __restrict__ grad_t)
{
    __shared__ double s_dz[kWave];
    const int b = blockIdx.y;
    if (threadIdx.x < kWave) s_dz[threadIdx.x] = threadIdx.x < ncls ? dz[(size_t)b * ncls + threadIdx.x] : 0.0;
    __syncthreads();
    const int e = blockIdx.x * kLiThreads + threadIdx.x;
    if (e >= E_max) return;
    const size_t at = (size_t)b * E_max + e;
    if (e >= clamp_count(ev_n[b], E_max)) {
        grad_t[at] = 0.0f;
        return;
    }
    const double dG = gk[at].y;
    double s = 0.0;
    if (dG != 0.0) {
        const float* row = WT + (size_t)clamp_src(ev_src[at], C_in) * ncls;
        for (int k = 0; k < ncls; ++k) s = fma((double)row[k], s_dz[k], s);
    }
    grad_t[at] = (float)(dG * s);
}

// grad_out_t[b][perm[b][j]] = grad_ev_t2[b][j] for the queue's events, 0 for
// every other spike slot.
__global__ __launch_bounds__(kLiThreads) void k_fill_f32(float* __restrict__ p, size_t n)
{
    const size_t i = (size_t)blockIdx.x * kLiThreads + threadIdx.x;
    if (i < n) p[i] = 0.0f;
}

__global__ __launch_bounds__(kLiThreads) void k_merge_grad(const float* __restrict__ g2,
                                                           const int32_t* __restrict__ perm,
                                                           const int32_t* __restrict__ ev_n2, int E2_max,
                                                           size_t per_sample, float* __restrict__ grad_out_t)
{
    const int b = blockIdx.y;
    const int j = blockIdx.x * kLiThreads + threadIdx.x;
    if (j >= clamp_count(ev_n2[b], E2_max)) return;
    const int p = perm[(size_t)b * E2_max + j];
    if (p >= 0 && (size_t)p < per_sample) grad_out_t[(size_t)b * per_sample + p] = g2[(size_t)b * E2_max + j];
}

struct LiLayout {
    size_t gk, z64, dz, loss_b, H, total;
};

static LiLayout li_layout(int B, int E_max, int C_in, int ncls)
{
    LiLayout L{};
    size_t off = 0;
    auto take = [&](size_t bytes) { size_t o = off; off += (bytes + 255) & ~(size_t)255; return o; };
    L.gk = take((size_t)B * E_max * sizeof(double2));
    L.z64 = take((size_t)B * ncls * sizeof(double));
    L.dz = take((size_t)B * ncls * sizeof(double));
    L.loss_b = take((size_t)B * sizeof(double));
    L.H = take((size_t)B * C_in * sizeof(unsigned long long));
    L.total = off + 256;
    return L;
}

static int check_li(const lif_li_params* q)
{
    if (!q) return LIF_ERR_ARG;
    if (!(q->tau_syn > 0.0) || !(q->tau_mem > q->tau_syn) || !isfinite(q->tau_mem)) return LIF_ERR_TAU;
    if (!(q->tau_li > 0.0)) return LIF_ERR_TAU;                     // +inf allowed: unweighted
    if (!(q->tau_max > 0.0) || !isfinite(q->tau_max) || !isfinite(q->beta)) return LIF_ERR_ARG;
    return LIF_OK;
}

}  // namespace lif

extern "C" size_t lif_li_readout_workspace_size(int B, int E_max, int C_in, int N_cls)
{
    if (B < 0 || E_max < 0 || C_in < 1 || N_cls < 1) return 0;
    return lif::li_layout(B, E_max, C_in, N_cls).total;
}

extern "C" int lif_li_readout(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                              const float* WT, int C_in, int N_cls, const lif_li_params* q,
                              const int32_t* labels, float* logits, float* loss, float* grad_WT,
                              float* grad_ev_t, void* ws, size_t ws_bytes, lif_stream_t stream_)
{
    using namespace lif;
    int rc = check_li(q);
    if (rc) return rc;
    if (B < 0 || E_max < 0 || C_in < 1 || N_cls < 1) return LIF_ERR_ARG;
    if (N_cls > LIF_LI_MAX_CLASSES) return LIF_ERR_SIZE;
    if ((size_t)C_in * (size_t)N_cls >= ((size_t)1 << 31) || (size_t)B * (size_t)E_max >= ((size_t)1 << 40))
        return LIF_ERR_SIZE;
    if (!WT || !ws || (B > 0 && !ev_n) || ((size_t)B * E_max > 0 && (!ev_t || !ev_src))) return LIF_ERR_ARG;
    if (!labels && (loss || grad_WT || grad_ev_t)) return LIF_ERR_ARG;
    const LiLayout L = li_layout(B, E_max, C_in, N_cls);
    if (ws_bytes < L.total) return LIF_ERR_WORKSPACE;
    hipStream_t stream = (hipStream_t)stream_;
    char* base = (char*)(((uintptr_t)ws + 255) & ~(uintptr_t)255);
    double2* gk = (double2*)(base + L.gk);
    double* z64 = (double*)(base + L.z64);
    double* dz = (double*)(base + L.dz);
    double* loss_b = (double*)(base + L.loss_b);
    unsigned long long* H = (unsigned long long*)(base + L.H);
    const LiModel m = make_li(*q);
    if (B == 0) {
        if (loss) TIMED_LAUNCH("li_loss", k_li_loss, dim3(1), dim3(1), 0, stream, loss_b, 0, loss);
        if (grad_WT) {
            const size_t n = (size_t)C_in * N_cls;
            TIMED_LAUNCH("li_fill", k_fill_f32, dim3((unsigned)((n + kLiThreads - 1) / kLiThreads)),
                         dim3(kLiThreads), 0, stream, grad_WT, n);
        }
        return check_launch();
    }
    const dim3 egrid((unsigned)((E_max + kLiThreads - 1) / kLiThreads > 0 ? (E_max + kLiThreads - 1) / kLiThreads : 1),
                     (unsigned)B);
    if (E_max > 0)
        TIMED_LAUNCH("li_kernel", k_li_kernel, egrid, dim3(kLiThreads), 0, stream, ev_t, ev_n, E_max, m, gk);
    TIMED_LAUNCH("li_logits", k_li_logits, dim3((unsigned)B, (unsigned)((N_cls + kWave - 1) / kWave)),
                 dim3(kLiThreads), 0, stream, ev_src, ev_n, E_max, WT, C_in, N_cls, gk, z64, logits);
    if (!labels) return check_launch();
    TIMED_LAUNCH("li_ce", k_li_ce, dim3((unsigned)B), dim3(kWave), 0, stream, z64, B, N_cls, labels, m.beta, dz,
                 loss_b);
    if (loss) TIMED_LAUNCH("li_loss", k_li_loss, dim3(1), dim3(1), 0, stream, loss_b, B, loss);
    if (grad_WT) {
        const size_t nh = (size_t)B * C_in;
        TIMED_LAUNCH("li_fill", k_fill_u64, dim3((unsigned)((nh + kLiThreads - 1) / kLiThreads)), dim3(kLiThreads),
                     0, stream, H, nh);
        if (E_max > 0)
            TIMED_LAUNCH("li_hist", k_li_hist, egrid, dim3(kLiThreads), 0, stream, ev_src, ev_n, E_max, C_in, gk, H);
        const size_t nw = (size_t)C_in * N_cls;
        TIMED_LAUNCH("li_grad_w", k_li_grad_w, dim3((unsigned)((nw + kLiThreads - 1) / kLiThreads)),
                     dim3(kLiThreads), 0, stream, H, B, C_in, N_cls, dz, grad_WT);
    }
    if (grad_ev_t && E_max > 0)
        TIMED_LAUNCH("li_grad_t", k_li_grad_t, egrid, dim3(kLiThreads), 0, stream, ev_src, ev_n, E_max, WT, C_in,
                     N_cls, gk, dz, grad_ev_t);
    return check_launch();
}

extern "C" int lif_merge_grad(const float* grad_ev_t2, const int32_t* perm, const int32_t* ev_n2, int B, int E2_max,
                              int N, int s_max, float* grad_out_t, lif_stream_t stream_)
{
    using namespace lif;
    if (B < 0 || E2_max < 0 || N < 1 || s_max < 1) return LIF_ERR_ARG;
    if (!grad_out_t || (B > 0 && !ev_n2) || ((size_t)B * E2_max > 0 && (!grad_ev_t2 || !perm))) return LIF_ERR_ARG;
    hipStream_t stream = (hipStream_t)stream_;
    const size_t per = (size_t)N * (size_t)s_max, n = (size_t)B * per;
    if (n)
        TIMED_LAUNCH("merge_grad_fill", k_fill_f32, dim3((unsigned)((n + kLiThreads - 1) / kLiThreads)),
                     dim3(kLiThreads), 0, stream, grad_out_t, n);
    if (B > 0 && E2_max > 0)
        TIMED_LAUNCH("merge_grad", k_merge_grad, dim3((unsigned)((E2_max + kLiThreads - 1) / kLiThreads), (unsigned)B),
                     dim3(kLiThreads), 0, stream, grad_ev_t2, perm, ev_n2, E2_max, per, grad_out_t);
    return check_launch();
}
