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
