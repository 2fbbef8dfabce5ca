// lif_api.hip -- host-side argument checks, model constants, version string
// and the optional per-kernel timer of liblif.so.
#include <mutex>
#include <string.h>
#include <vector>

#include "lif_host.hpp"

namespace lif {

int check_params(const lif_params* p)
{
    if (!p) return LIF_ERR_ARG;
    if (!(p->tau_syn > 0.0) || !(p->tau_mem > p->tau_syn) || !isfinite(p->tau_mem)) return LIF_ERR_TAU;
    // The neuron rests at V = 0 below its threshold: 0 < v_th, v_reset < v_th.
    if (!(p->v_reset < p->v_th) || !(p->v_th > 0.0) || !isfinite(p->v_th) || !isfinite(p->v_reset))
        return LIF_ERR_THRESHOLD;
    if (p->s_max < 1) return LIF_ERR_ARG;
    if (isnan(p->t_end) || !(p->solver_reg >= 0.0)) return LIF_ERR_ARG;
    if (p->reserved != 0 || (p->flags & ~(LIF_VALIDATE | LIF_ROOT_GENERAL))) return LIF_ERR_ARG;
    return LIF_OK;
}

Model make_model(const lif_params& p)
{
    Model m{};
    m.tm = p.tau_mem;
    m.ts = p.tau_syn;
    m.th = p.v_th;
    m.vr = p.v_reset;
    m.t_end = p.t_end;
    m.kappa = p.tau_syn / (p.tau_mem - p.tau_syn);
    m.inv_tm = 1.0 / p.tau_mem;
    m.inv_ts = 1.0 / p.tau_syn;
    m.a_rate = m.inv_ts - m.inv_tm;
    m.c_tv = p.tau_mem * p.tau_syn / (p.tau_mem - p.tau_syn);
    m.t_peak = m.c_tv * log(p.tau_mem / p.tau_syn);
    // The no-crossing screen is evaluated in float64 with relative error
    // ~1e-15; the margin keeps it conservative.
    m.th_lo = p.v_th - 1e-9 * fmax(1.0, fabs(p.v_th));
    m.thk_lo = m.th_lo / m.kappa;
    m.inv_ktm = 1.0 / (m.kappa * p.tau_mem);
    m.inv_th = 1.0 / p.v_th;
    m.th_1k = p.v_th * (1.0 + m.kappa);
    m.ts_tm = p.tau_syn / p.tau_mem;
    m.dth = p.v_th - p.v_reset;
    m.f_th = (float)m.th;
    m.f_inv_tm = (float)m.inv_tm;
    m.reg = p.solver_reg;
    // tau_m / tau_s = p + 1 exactly for an integer 1 <= p <= 4: the
    // spike-time solve works on a polynomial (root_poly)
    m.p_int = 0;
    for (int q = 1; q <= 4; ++q)
        if (p.tau_mem / p.tau_syn == (double)(q + 1)) m.p_int = q;
    if (p.flags & LIF_ROOT_GENERAL) m.p_int = 0;
    m.s_max = p.s_max;
    m.flags = p.flags;
    return m;
}

int validate_forward_args(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                          const float* WT, int C_in, int N, const lif_params* p, const float* out_t,
                          const int32_t* out_n, const int32_t* status)
{
    int rc = check_params(p);
    if (rc) return rc;
    if (B < 0 || E_max < 0 || C_in < 1 || N < 1) return LIF_ERR_ARG;
    if (!WT || !out_t || !out_n || !status) return LIF_ERR_ARG;
    if (B > 0 && !ev_n) return LIF_ERR_ARG;
    if ((size_t)B * (size_t)E_max > 0 && (!ev_t || !ev_src)) return LIF_ERR_ARG;
    if ((size_t)B * (size_t)E_max >= ((size_t)1 << 40)) return LIF_ERR_SIZE;
    // the walks address W^T through a buffer descriptor with a 32-bit byte range
    if ((size_t)C_in * (size_t)N >= ((size_t)1 << 29)) return LIF_ERR_SIZE;
    return LIF_OK;
}

int check_launch()
{
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? LIF_OK : LIF_ERR_HIP;
}

// ---------------------------------------------------------------------------
// Kernel timer
// ---------------------------------------------------------------------------
namespace {
struct TimerRec {
    const char* name;
    hipEvent_t a, b;
};
std::mutex g_mu;
bool g_on = false;
std::vector<TimerRec> g_recs;
std::vector<hipEvent_t> g_pool;
size_t g_pool_used = 0;

hipEvent_t pool_get()
{
    if (g_pool_used == g_pool.size()) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) return nullptr;
        g_pool.push_back(e);
    }
    return g_pool[g_pool_used++];
}
}  // namespace

bool timer_on() { return g_on; }

bool timer_events(const char* name, hipEvent_t* start, hipEvent_t* stop)
{
    std::lock_guard<std::mutex> lk(g_mu);
    hipEvent_t a = pool_get(), b = pool_get();
    if (!a || !b) return false;
    g_recs.push_back({name, a, b});
    *start = a;
    *stop = b;
    return true;
}

}  // namespace lif

extern "C" const char* lif_version(void)
{
    return "liblif 0.1.0 (gfx950, float64 state, segment scan + resolve)";
}

extern "C" void lif_timer_enable(int on)
{
    std::lock_guard<std::mutex> lk(lif::g_mu);
    lif::g_recs.clear();
    lif::g_pool_used = 0;
    lif::g_on = on != 0;
}

extern "C" int lif_timer_read(const char** names, double* total_ms, int32_t* launches, int cap)
{
    std::lock_guard<std::mutex> lk(lif::g_mu);
    std::vector<const char*> nm;
    std::vector<double> ms;
    std::vector<int32_t> cnt;
    for (auto& r : lif::g_recs) {
        (void)hipEventSynchronize(r.b);
        float t = 0.0f;
        (void)hipEventElapsedTime(&t, r.a, r.b);
        size_t j = 0;
        for (; j < nm.size(); ++j)
            if (strcmp(nm[j], r.name) == 0) break;
        if (j == nm.size()) { nm.push_back(r.name); ms.push_back(0.0); cnt.push_back(0); }
        ms[j] += t;
        cnt[j] += 1;
    }
    for (size_t j = 0; j < nm.size() && (int)j < cap; ++j) {
        if (names) names[j] = nm[j];
        if (total_ms) total_ms[j] = ms[j];
        if (launches) launches[j] = cnt[j];
    }
    return (int)nm.size();
}
