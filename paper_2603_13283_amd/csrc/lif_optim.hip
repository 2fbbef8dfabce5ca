// lif_optim.hip -- the optimiser step of training (App. E: models are
// trained with Adam, Kingma & Ba): one elementwise update per parameter,
// moments and the bias-corrected step in float64, parameters and moments
// stored in float32.
#include "lif_common.hpp"
#include "lif_host.hpp"

namespace lif {

constexpr int kAdamThreads = 256;

__global__ __launch_bounds__(kAdamThreads) void k_adam(float* __restrict__ p, const float* __restrict__ g,
                                                       float* __restrict__ m1, float* __restrict__ m2, size_t n,
                                                       double lr, double b1, double b2, double eps, double c1,
                                                       double c2)
{
    const size_t i = (size_t)blockIdx.x * kAdamThreads + threadIdx.x;
    if (i >= n) return;
    const double gi = (double)g[i];
    const double a = b1 * (double)m1[i] + (1.0 - b1) * gi;
    const double v = b2 * (double)m2[i] + (1.0 - b2) * gi * gi;
    m1[i] = (float)a;
    m2[i] = (float)v;
    p[i] = (float)((double)p[i] - lr * (a / c1) / (sqrt(v / c2) + eps));
}

}  // namespace lif

extern "C" int lif_adam_step(float* param, const float* grad, float* m1, float* m2, size_t n,
                             const lif_adam_params* a, int step, lif_stream_t stream)
{
    using namespace lif;
    if (!a || step < 1 || (n > 0 && (!param || !grad || !m1 || !m2))) return LIF_ERR_ARG;
    if (!(a->lr >= 0.0) || !(a->beta1 >= 0.0 && a->beta1 < 1.0) || !(a->beta2 >= 0.0 && a->beta2 < 1.0) ||
        !(a->eps > 0.0))
        return LIF_ERR_ARG;
    if (n == 0) return LIF_OK;
    const double c1 = 1.0 - pow(a->beta1, (double)step), c2 = 1.0 - pow(a->beta2, (double)step);
    TIMED_LAUNCH("adam", k_adam, dim3((unsigned)((n + kAdamThreads - 1) / kAdamThreads)), dim3(kAdamThreads), 0,
                 (hipStream_t)stream, param, grad, m1, m2, n, a->lr, a->beta1, a->beta2, a->eps, c1, c2);
    return check_launch();
}

// ---------------------------------------------------------------------------
// Two elementwise pieces of the training step: y += x (adding the direct
// part of a regulariser gradient to a layer's gradient), and the delay
// activation d = softplus(x) = log(1 + e^{beta x}) / beta (App. E.5) with its
// derivative sigmoid(beta x).
// ---------------------------------------------------------------------------
namespace lif {

__global__ __launch_bounds__(kAdamThreads) void k_add(float* __restrict__ y, const float* __restrict__ x, size_t n)
{
    const size_t i = (size_t)blockIdx.x * kAdamThreads + threadIdx.x;
    if (i < n) y[i] += x[i];
}

// log(1 + e^z) without overflow: max(z, 0) + log1p(e^{-|z|}).
__global__ __launch_bounds__(kAdamThreads) void k_softplus(const float* __restrict__ x, float* __restrict__ d,
                                                           size_t n, double beta)
{
    const size_t i = (size_t)blockIdx.x * kAdamThreads + threadIdx.x;
    if (i >= n) return;
    const double z = beta * (double)x[i];
    d[i] = (float)((fmax(z, 0.0) + log1p(exp(-fabs(z)))) / beta);
}

// g_x = g_d sigmoid(beta x), the sigmoid as e^{min(z,0)} / (1 + e^{-|z|}).
__global__ __launch_bounds__(kAdamThreads) void k_softplus_grad(const float* __restrict__ x,
                                                                const float* __restrict__ gd, float* __restrict__ gx,
                                                                size_t n, double beta)
{
    const size_t i = (size_t)blockIdx.x * kAdamThreads + threadIdx.x;
    if (i >= n) return;
    const double z = beta * (double)x[i];
    gx[i] = (float)((double)gd[i] * exp(fmin(z, 0.0)) / (1.0 + exp(-fabs(z))));
}

static dim3 elementwise_grid(size_t n) { return dim3((unsigned)((n + kAdamThreads - 1) / kAdamThreads)); }

}  // namespace lif

extern "C" int lif_add(float* y, const float* x, size_t n, lif_stream_t stream)
{
    using namespace lif;
    if (n > 0 && (!y || !x)) return LIF_ERR_ARG;
    if (n == 0) return LIF_OK;
    if ((n + kAdamThreads - 1) / kAdamThreads > 0x7fffffffull) return LIF_ERR_SIZE;
    TIMED_LAUNCH("add", k_add, elementwise_grid(n), dim3(kAdamThreads), 0, (hipStream_t)stream, y, x, n);
    return check_launch();
}

extern "C" int lif_softplus(const float* x, float* d, size_t n, double beta, lif_stream_t stream)
{
    using namespace lif;
    if ((n > 0 && (!x || !d)) || !(beta > 0.0) || !isfinite(beta)) return LIF_ERR_ARG;
    if (n == 0) return LIF_OK;
    if ((n + kAdamThreads - 1) / kAdamThreads > 0x7fffffffull) return LIF_ERR_SIZE;
    TIMED_LAUNCH("softplus", k_softplus, elementwise_grid(n), dim3(kAdamThreads), 0, (hipStream_t)stream, x, d, n,
                 beta);
    return check_launch();
}

extern "C" int lif_softplus_grad(const float* x, const float* grad_d, float* grad_x, size_t n, double beta,
                                 lif_stream_t stream)
{
    using namespace lif;
    if ((n > 0 && (!x || !grad_d || !grad_x)) || !(beta > 0.0) || !isfinite(beta)) return LIF_ERR_ARG;
    if (n == 0) return LIF_OK;
    if ((n + kAdamThreads - 1) / kAdamThreads > 0x7fffffffull) return LIF_ERR_SIZE;
    TIMED_LAUNCH("softplus_grad", k_softplus_grad, elementwise_grid(n), dim3(kAdamThreads), 0, (hipStream_t)stream, x,
                 grad_d, grad_x, n, beta);
    return check_launch();
}
