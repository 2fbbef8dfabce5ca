/*
 * lif_oracle.c -- float64 CPU oracle for the event-driven current-based LIF
 * layer with exact hard reset ("Bullet Trains", arXiv 2603.13283).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, sequential
 * reference that the GPU path is checked against.  Only the test suite, the
 * smoke check and the CPU-baseline leg of the benchmark may load it.  It
 * shares no code, header, table or constant generator with the GPU library.
 *
 * Every (sample, neuron) pair is simulated independently, one event at a
 * time, exactly as the paper's serial semantics describe (Sec. 4 baseline,
 * Appendix E.2 and E.3): before each input event the neuron checks whether
 * it fires in the interval up to that event (Sec. 3.2.2 interval rule); if so
 * the spike time is solved, the voltage is hard-reset and the same interval
 * is tested again from the spike time.  All arithmetic is IEEE float64 on the
 * float32 input values widened to float64.
 *
 * Readings where the paper is silent (each is also listed in the design
 * notes of the repository):
 *   - the neuron starts at V = 0, I = 0 at t = 0;
 *   - the reset acts on V only; I keeps decaying (Eq. curr_dyn);
 *   - the threshold test is V >= V_th;
 *   - an interior maximum needs I0 > V0 *and* D = V0 (tm - ts) + I0 ts > 0,
 *     otherwise the log argument of Eq. t_vmax is not > 1;
 *   - the root bracket is [0, min(t_Vmax, interval length)];
 *   - the root is the smallest float64 offset tau with V(tau) >= V_th;
 *   - the interval after the last event extends to t_end (default +inf);
 *   - after the s_max-th spike the neuron stops (it is reported as capped).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <pthread.h>

typedef struct {
    double tau_mem;    /* membrane time constant tau_m (s)                   */
    double tau_syn;    /* synaptic time constant tau_s (s), tau_s < tau_m    */
    double v_th;       /* threshold V_th                                     */
    double v_reset;    /* reset potential V_reset                            */
    double t_end;      /* end of the last interval (+inf: unbounded)         */
    int32_t s_max;     /* output spike capacity per neuron                   */
    double solver_reg; /* backward: floor on dV/dt at a spike (0: off)       */
    double tie_band;   /* |V_max - V_th| below this marks a near-tie         */
} or_params;

/* ---------------------------------------------------------------------- */
/* Closed-form sub-threshold solution (Appendix A, Eq. mem_pot and curr).  */
/* ---------------------------------------------------------------------- */

static double kappa(const or_params* p) { return p->tau_syn / (p->tau_mem - p->tau_syn); }

/* V(t) from (V0, I0) after time t >= 0 (Eq. mem_pot). */
static double v_at(const or_params* p, double V0, double I0, double t)
{
    if (isinf(t)) return 0.0;
    double em = exp(-t / p->tau_mem), es = exp(-t / p->tau_syn);
    return V0 * em + I0 * kappa(p) * (em - es);
}

/* I(t) from I0 after time t (Eq. curr). */
static double i_at(const or_params* p, double I0, double t)
{
    if (isinf(t)) return 0.0;
    return I0 * exp(-t / p->tau_syn);
}

/* dV/dt from the ODE itself (Eq. mem_dyn): tau_m dV/dt = -V + I. */
static double dvdt(const or_params* p, double V, double I) { return (I - V) / p->tau_mem; }

/* ---------------------------------------------------------------------- */
/* Interval check (Sec. 3.2.2 rule; t_Vmax from Appendix D.1, Eq. t_vmax). */
/* ---------------------------------------------------------------------- */

typedef struct {
    int crossing;    /* 1 if V reaches V_th inside (0, len]                 */
    double hi;       /* right end of the root bracket: min(t_Vmax, len)     */
    double vmax;     /* maximum of V over [0, len] (for the near-tie flag)  */
} or_check;

static or_check check_interval(const or_params* p, double V0, double I0, double len)
{
    or_check r = {0, len, V0};
    double vend = v_at(p, V0, I0, len);
    if (vend > r.vmax) r.vmax = vend;
    /* Interior maximum: dV/dt = 0 has its root at Eq. t_vmax when the log
     * argument I0 tm / (V0 (tm - ts) + I0 ts) exceeds 1. */
    double D = V0 * (p->tau_mem - p->tau_syn) + I0 * p->tau_syn;
    int has_max = (I0 > V0) && (D > 0.0);
    double tv = INFINITY;
    if (has_max) {
        tv = (p->tau_mem * p->tau_syn / (p->tau_mem - p->tau_syn)) * log(I0 * p->tau_mem / D);
        if (tv < len) {
            double vv = v_at(p, V0, I0, tv);
            if (vv > r.vmax) r.vmax = vv;
        }
    }
    /* The literal rule: a spike if V(t_next) >= V_th, or if t_Vmax lies in the
     * interval and V(t_Vmax) >= V_th. */
    if (vend >= p->v_th) {
        r.crossing = 1;
        r.hi = has_max && tv < len ? tv : len;
    } else if (has_max && tv < len && v_at(p, V0, I0, tv) >= p->v_th) {
        r.crossing = 1;
        r.hi = tv;
    }
    return r;
}

/* ---------------------------------------------------------------------- */
/* Spike-time root (Appendix D.1 Newton-Raphson, bracketed and clamped to   */
/* the search interval; D.2 bisection as the fallback step).                */
/* ---------------------------------------------------------------------- */

/* Smallest float64 tau in (0, hi] with V(tau) >= V_th, where V(hi) >= V_th
 * and V is increasing on [0, hi]. */
static double solve_root(const or_params* p, double V0, double I0, double hi)
{
    const double hi0 = hi;
    double lo = 0.0;
    double t = 0.5 * hi;                      /* t0 = t_Vmax / 2 (App. D.1) */
    for (int it = 0; it < 200; ++it) {
        double v = v_at(p, V0, I0, t);
        if (v >= p->v_th) hi = t; else lo = t;
        double d = dvdt(p, v, i_at(p, I0, t));
        double tn = (d > 0.0) ? t - (v - p->v_th) / d : 0.5 * (lo + hi);
        if (!(tn > lo && tn < hi)) tn = 0.5 * (lo + hi);   /* clamp: bisect */
        if (tn == t || hi - lo <= 2.0 * (nextafter(hi, INFINITY) - hi)) break;
        t = tn;
    }
    /* Polish to the smallest float64 with V >= V_th: step up from the last
     * iterate until the threshold is met, then down while it still is. */
    double r = t;
    for (int it = 0; it < 256 && r < hi0 && v_at(p, V0, I0, r) < p->v_th; ++it)
        r = nextafter(r, INFINITY);
    if (v_at(p, V0, I0, r) < p->v_th) r = hi;        /* bracket end satisfies it */
    for (int it = 0; it < 256; ++it) {
        double q = nextafter(r, 0.0);
        if (q <= 0.0 || v_at(p, V0, I0, q) < p->v_th) break;
        r = q;
    }
    return r;
}

/* ---------------------------------------------------------------------- */
/* Forward: one neuron, serial event loop with restart after each spike.    */
/* ---------------------------------------------------------------------- */

typedef struct {
    int32_t n_spikes;
    int32_t capped;
    double tie_t;       /* start time of the first near-tie interval (+inf) */
    double min_gap;     /* min over checked intervals of |V_max - V_th|     */
} or_neuron_result;

static or_neuron_result simulate_neuron(const or_params* p, const float* ev_t, const int32_t* ev_src,
                                        int n, const float* WT, int N, int i,
                                        double* st, double* si, int32_t* sk)
{
    or_neuron_result res = {0, 0, INFINITY, INFINITY};
    double t_cur = 0.0, V = 0.0, I = 0.0;
    int k = 0;
    for (;;) {
        double t_hi = (k < n) ? (double)ev_t[k] : p->t_end;
        double len = t_hi - t_cur;
        if (len > 0.0) {
            or_check c = check_interval(p, V, I, len);
            double gap = fabs(c.vmax - p->v_th);
            if (gap < res.min_gap) res.min_gap = gap;
            if (gap < p->tie_band && t_cur < res.tie_t) res.tie_t = t_cur;
            if (c.crossing) {
                double tau = solve_root(p, V, I, c.hi);
                double Istar = i_at(p, I, tau);
                st[res.n_spikes] = t_cur + tau;
                si[res.n_spikes] = Istar;
                sk[res.n_spikes] = k;          /* events 0 .. k-1 came before this spike */
                res.n_spikes++;
                if (res.n_spikes >= p->s_max) { res.capped = 1; return res; }
                /* Hard reset of V only; the interval is tested again from t*. */
                V = p->v_reset;
                I = Istar;
                t_cur = t_cur + tau;
                continue;
            }
        }
        if (k >= n) break;
        /* Eq. affine: s_k = M(dt) s_{k-1} + (0, w). */
        if (len > 0.0) {
            double Vn = v_at(p, V, I, len);
            I = i_at(p, I, len);
            V = Vn;
        }
        I += (double)WT[(size_t)ev_src[k] * (size_t)N + (size_t)i];
        t_cur = t_hi;
        ++k;
    }
    return res;
}

/* Work split over (sample, neuron) items with plain pthreads. */
typedef struct {
    const or_params* p;
    const float* ev_t; const int32_t* ev_src; const int32_t* ev_n;
    int B, E_max; const float* WT; int C_in, N;
    double* out_t; double* out_i; int32_t* out_k; int32_t* out_n; int32_t* capped; double* tie_t;
    double* min_gap;
    int tid, nthreads;
} fwd_job;

static void* fwd_worker(void* arg)
{
    fwd_job* j = (fwd_job*)arg;
    size_t total = (size_t)j->B * (size_t)j->N;
    for (size_t item = (size_t)j->tid; item < total; item += (size_t)j->nthreads) {
        int b = (int)(item / (size_t)j->N), i = (int)(item % (size_t)j->N);
        size_t o = item * (size_t)j->p->s_max;
        for (int s = 0; s < j->p->s_max; ++s) {
            j->out_t[o + s] = INFINITY;
            j->out_i[o + s] = 0.0;
            j->out_k[o + s] = 0;
        }
        or_neuron_result r = simulate_neuron(j->p, j->ev_t + (size_t)b * j->E_max,
                                             j->ev_src + (size_t)b * j->E_max, j->ev_n[b],
                                             j->WT, j->N, i, j->out_t + o, j->out_i + o, j->out_k + o);
        j->out_n[item] = r.n_spikes;
        j->capped[item] = r.capped;
        j->tie_t[item] = r.tie_t;
        j->min_gap[item] = r.min_gap;
    }
    return NULL;
}

static int run_threads(void* (*fn)(void*), void* jobs, size_t job_size, int nthreads)
{
    pthread_t* th = (pthread_t*)malloc(sizeof(pthread_t) * (size_t)nthreads);
    if (!th) return -1;
    for (int t = 0; t < nthreads; ++t)
        pthread_create(&th[t], NULL, fn, (char*)jobs + (size_t)t * job_size);
    for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
    free(th);
    return 0;
}

/* Forward over a batch.  Outputs are [B][N][s_max] (times, I at spike, and
 * the number of input events consumed before each spike; +inf, 0 and 0
 * padding), [B][N] counts, capped flags, first near-tie interval start and
 * the smallest |V_max - V_th| seen. */
int or_forward(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
               const float* WT, int C_in, int N, const or_params* p, int nthreads,
               double* out_t, double* out_i, int32_t* out_k, int32_t* out_n, int32_t* capped,
               double* tie_t, double* min_gap)
{
    if (!(p->tau_mem > p->tau_syn && p->tau_syn > 0.0) || !(p->v_reset < p->v_th) || p->s_max < 1)
        return -1;
    if (nthreads < 1) nthreads = 1;
    fwd_job* jobs = (fwd_job*)calloc((size_t)nthreads, sizeof(fwd_job));
    if (!jobs) return -2;
    for (int t = 0; t < nthreads; ++t) {
        fwd_job j = {p, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N,
                     out_t, out_i, out_k, out_n, capped, tie_t, min_gap, t, nthreads};
        jobs[t] = j;
    }
    int rc = run_threads(fwd_worker, jobs, sizeof(fwd_job), nthreads);
    free(jobs);
    return rc;
}

/* ---------------------------------------------------------------------- */
/* Chunk mode (Sec. 3.2.1 "Speculative execution" and "Fixed compute        */
/* budget", Appendix E.2): the neuron takes its queue K events at a time.   */
/* Each chunk iteration tests the intervals closed by its events in order   */
/* (and, in the chunk that holds the last event, the interval after it up   */
/* to t_end); at the first crossing it commits one spike, hard-resets, and  */
/* the next iteration starts at the spike time with the same pending event  */
/* (the chunk's later events are processed but discarded); without a        */
/* crossing all its events are consumed.  At most C iterations run and at   */
/* most s_max spikes are kept.  Work counters (Appendix G): processed = the */
/* events of every iteration's chunk (an event visited twice counts twice), */
/* consumed = the events consumed when the neuron stops.                    */
/* ---------------------------------------------------------------------- */
static or_neuron_result simulate_neuron_chunked(const or_params* p, const float* ev_t, const int32_t* ev_src, int n,
                                                const float* WT, int N, int i, int K, int C, double* st, double* si,
                                                int32_t* sk, int32_t* consumed, int32_t* processed)
{
    or_neuron_result res = {0, 0, INFINITY, INFINITY};
    double t_cur = 0.0, V = 0.0, I = 0.0;
    int k = 0, chunks = 0;
    long long work = 0;
    int finished = 0;
    while (!finished && !res.capped && chunks < C) {
        ++chunks;
        const int end = (k + K < n) ? k + K : n;
        work += end - k;
        for (;;) {
            double t_hi;
            if (k < end) t_hi = (double)ev_t[k];
            else if (end == n) t_hi = p->t_end;      /* the interval after the last event */
            else break;                              /* the chunk is consumed */
            double len = t_hi - t_cur;
            if (len > 0.0) {
                or_check c = check_interval(p, V, I, len);
                double gap = fabs(c.vmax - p->v_th);
                if (gap < res.min_gap) res.min_gap = gap;
                if (gap < p->tie_band && t_cur < res.tie_t) res.tie_t = t_cur;
                if (c.crossing) {
                    double tau = solve_root(p, V, I, c.hi);
                    double Istar = i_at(p, I, tau);
                    st[res.n_spikes] = t_cur + tau;
                    si[res.n_spikes] = Istar;
                    sk[res.n_spikes] = k;
                    res.n_spikes++;
                    if (res.n_spikes >= p->s_max) res.capped = 1;
                    V = p->v_reset;
                    I = Istar;
                    t_cur = t_cur + tau;
                    break;                           /* the next iteration restarts here */
                }
            }
            if (k >= n) { finished = 1; break; }     /* the last interval holds no spike */
            if (len > 0.0) {
                double Vn = v_at(p, V, I, len);
                I = i_at(p, I, len);
                V = Vn;
            }
            I += (double)WT[(size_t)ev_src[k] * (size_t)N + (size_t)i];
            t_cur = t_hi;
            ++k;
        }
    }
    *consumed = k;
    *processed = (int32_t)work;
    return res;
}

typedef struct {
    fwd_job f;
    int K, C;
    int32_t* consumed; int32_t* processed;
} chunk_job;

static void* chunk_worker(void* arg)
{
    chunk_job* cj = (chunk_job*)arg;
    fwd_job* j = &cj->f;
    size_t total = (size_t)j->B * (size_t)j->N;
    for (size_t item = (size_t)j->tid; item < total; item += (size_t)j->nthreads) {
        int b = (int)(item / (size_t)j->N), i = (int)(item % (size_t)j->N);
        size_t o = item * (size_t)j->p->s_max;
        for (int s = 0; s < j->p->s_max; ++s) {
            j->out_t[o + s] = INFINITY;
            j->out_i[o + s] = 0.0;
            j->out_k[o + s] = 0;
        }
        or_neuron_result r = simulate_neuron_chunked(j->p, j->ev_t + (size_t)b * j->E_max,
                                                     j->ev_src + (size_t)b * j->E_max, j->ev_n[b], j->WT, j->N, i,
                                                     cj->K, cj->C, j->out_t + o, j->out_i + o, j->out_k + o,
                                                     cj->consumed + item, cj->processed + item);
        j->out_n[item] = r.n_spikes;
        j->capped[item] = r.capped;
        j->tie_t[item] = r.tie_t;
        j->min_gap[item] = r.min_gap;
    }
    return NULL;
}

/* Chunk-mode forward over a batch (outputs as or_forward, plus the
 * per-(sample, neuron) consumed and processed event counts). */
int or_forward_chunked(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                       const float* WT, int C_in, int N, const or_params* p, int K, int C, int nthreads,
                       double* out_t, double* out_i, int32_t* out_k, int32_t* out_n, int32_t* capped,
                       double* tie_t, double* min_gap, int32_t* consumed, int32_t* processed)
{
    if (!(p->tau_mem > p->tau_syn && p->tau_syn > 0.0) || !(p->v_reset < p->v_th) || p->s_max < 1 || K < 1 || C < 1)
        return -1;
    if (nthreads < 1) nthreads = 1;
    chunk_job* jobs = (chunk_job*)calloc((size_t)nthreads, sizeof(chunk_job));
    if (!jobs) return -2;
    for (int t = 0; t < nthreads; ++t) {
        fwd_job j = {p, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N,
                     out_t, out_i, out_k, out_n, capped, tie_t, min_gap, t, nthreads};
        jobs[t].f = j;
        jobs[t].K = K;
        jobs[t].C = C;
        jobs[t].consumed = consumed;
        jobs[t].processed = processed;
    }
    int rc = run_threads(chunk_worker, jobs, sizeof(chunk_job), nthreads);
    free(jobs);
    return rc;
}

/* Membrane trace of one neuron right after every input event (no spikes
 * beyond what the full forward finds); used by the closed-form pins.
 * V_after[k], I_after[k] are the true (reset-including) state just after
 * event k. */
int or_trace(const float* ev_t, const int32_t* ev_src, int n, const float* WT, int N, int i,
             const or_params* p, double* V_after, double* I_after)
{
    double t_cur = 0.0, V = 0.0, I = 0.0;
    int k = 0, ns = 0;
    for (;;) {
        double t_hi = (k < n) ? (double)ev_t[k] : p->t_end;
        double len = t_hi - t_cur;
        if (len > 0.0 && ns < p->s_max) {
            or_check c = check_interval(p, V, I, len);
            if (c.crossing) {
                double tau = solve_root(p, V, I, c.hi);
                I = i_at(p, I, tau);
                V = p->v_reset;
                t_cur += tau;
                ++ns;
                continue;
            }
        }
        if (k >= n) break;
        if (len > 0.0) {
            double Vn = v_at(p, V, I, len);
            I = i_at(p, I, len);
            V = Vn;
        }
        I += (double)WT[(size_t)ev_src[k] * (size_t)N + (size_t)i];
        t_cur = t_hi;
        V_after[k] = V;
        I_after[k] = I;
        ++k;
    }
    return ns;
}

/* ---------------------------------------------------------------------- */
/* Backward (Appendix D.3 implicit differentiation, chained through the     */
/* hard resets).                                                            */
/*                                                                          */
/* With the resets written as subtractions, spike s satisfies              */
/*   F_s = sum_{k: t_k < t_s} w_k K(t_s - t_k)                              */
/*         - (V_th - V_reset) sum_{s' < s} exp(-(t_s - t_s')/tm) - V_th = 0 */
/* with K(u) = kappa (exp(-u/tm) - exp(-u/ts)).  The implicit function      */
/* theorem (Eq. ift_vjp) gives dt_s = -(dF_s/dt_s)^-1 dF_s, where           */
/* dF_s/dt_s = dV/dt at the spike = (I(t_s) - V_th)/tm (Eq. mem_dyn),       */
/* floored by the solver regularisation.  The adjoints are taken by a       */
/* reverse pass over the spikes of each neuron, then every input event      */
/* collects its weight and time gradients directly from the sums.           */
/*                                                                          */
/* Which events a spike depends on is the forward pass's own decision: the  */
/* spike solved in the interval before event k depends on events 0 .. k-1   */
/* (out_k holds k).  An event at exactly the spike time comes after it (the */
/* interval is tested before its closing event is consumed).  Deciding this */
/* from the index instead of comparing times keeps the decision when the    */
/* spike times handed over have been rounded (to float32, a spike can round */
/* onto the time of the event just before it); the offset t_s - t_k is then */
/* at least 0.                                                              */
/* ---------------------------------------------------------------------- */

typedef struct {
    const or_params* p;
    const float* ev_t; const int32_t* ev_src; const int32_t* ev_n;
    int B, E_max; const float* WT; int C_in, N;
    const double* out_t; const double* out_i; const int32_t* out_k; const int32_t* out_n;
    const double* grad_out_t;
    double* gW_part;   /* [nthreads][C_in][N] partial weight gradients       */
    double* gT_part;   /* [nthreads][B][E_max] partial time gradients        */
    int tid, nthreads;
} bwd_job;

static void* bwd_worker(void* arg)
{
    bwd_job* j = (bwd_job*)arg;
    const or_params* p = j->p;
    const double tm = p->tau_mem, ts = p->tau_syn, ka = kappa(p);
    const int smax = p->s_max;
    double* mu = (double*)malloc(sizeof(double) * (size_t)smax);
    double* gW = j->gW_part + (size_t)j->tid * (size_t)j->C_in * (size_t)j->N;
    double* gT = j->gT_part + (size_t)j->tid * (size_t)j->B * (size_t)j->E_max;
    size_t total = (size_t)j->B * (size_t)j->N;
    for (size_t item = (size_t)j->tid; item < total; item += (size_t)j->nthreads) {
        int b = (int)(item / (size_t)j->N), i = (int)(item % (size_t)j->N);
        int ns = j->out_n[item];
        if (ns <= 0) continue;
        const double* ts_ = j->out_t + item * (size_t)smax;
        const double* is_ = j->out_i + item * (size_t)smax;
        const int32_t* ks_ = j->out_k + item * (size_t)smax;
        const double* g = j->grad_out_t + item * (size_t)smax;
        /* Reverse pass over the spikes: lambda_s = dL/dt_s (total),
         * mu_s = -lambda_s / V'_s is the multiplier of constraint F_s. */
        for (int s = ns - 1; s >= 0; --s) {
            double lam = g[s];
            for (int s2 = s + 1; s2 < ns; ++s2)
                lam -= (p->v_th - p->v_reset) / tm * mu[s2] * exp(-(ts_[s2] - ts_[s]) / tm);
            double vp = dvdt(p, p->v_th, is_[s]);
            if (vp < p->solver_reg) vp = p->solver_reg;
            mu[s] = -lam / vp;
        }
        /* Each event before a spike: dF_s/dw_src = K(t_s - t_k),
         * dF_s/dt_k = -w K'(t_s - t_k). */
        const float* et = j->ev_t + (size_t)b * j->E_max;
        const int32_t* es = j->ev_src + (size_t)b * j->E_max;
        int n = j->ev_n[b];
        for (int k = 0; k < n; ++k) {
            if (k >= ks_[ns - 1]) break;          /* no spike depends on event k */
            double tk = (double)et[k];
            double a = 0.0, ad = 0.0;
            for (int s = 0; s < ns; ++s) {
                if (k >= ks_[s]) continue;        /* spike s came before event k */
                double u = ts_[s] - tk;
                if (u < 0.0) u = 0.0;
                double em = exp(-u / tm), es2 = exp(-u / ts);
                a += mu[s] * ka * (em - es2);
                ad += mu[s] * ka * (-em / tm + es2 / ts);
            }
            double w = (double)j->WT[(size_t)es[k] * (size_t)j->N + (size_t)i];
            gW[(size_t)es[k] * (size_t)j->N + (size_t)i] += a;
            gT[(size_t)b * j->E_max + k] += -w * ad;
        }
    }
    free(mu);
    return NULL;
}

/* Backward over a batch: grad_WT [C_in][N] and grad_ev_t [B][E_max] are
 * overwritten.  out_t/out_i/out_k/out_n are forward outputs for the same
 * inputs (the oracle's own, possibly rounded). */
int or_backward(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                const float* WT, int C_in, int N, const or_params* p, int nthreads,
                const double* out_t, const double* out_i, const int32_t* out_k, const int32_t* out_n,
                const double* grad_out_t, double* grad_WT, double* grad_ev_t)
{
    if (nthreads < 1) nthreads = 1;
    size_t wsz = (size_t)C_in * (size_t)N, tsz = (size_t)B * (size_t)E_max;
    double* gW_part = (double*)calloc(wsz * (size_t)nthreads, sizeof(double));
    double* gT_part = (double*)calloc(tsz * (size_t)nthreads, sizeof(double));
    bwd_job* jobs = (bwd_job*)calloc((size_t)nthreads, sizeof(bwd_job));
    if (!gW_part || !gT_part || !jobs) { free(gW_part); free(gT_part); free(jobs); return -2; }
    for (int t = 0; t < nthreads; ++t) {
        bwd_job j = {p, ev_t, ev_src, ev_n, B, E_max, WT, C_in, N, out_t, out_i, out_k, out_n, grad_out_t,
                     gW_part, gT_part, t, nthreads};
        jobs[t] = j;
    }
    run_threads(bwd_worker, jobs, sizeof(bwd_job), nthreads);
    for (size_t x = 0; x < wsz; ++x) {
        double s = 0.0;
        for (int t = 0; t < nthreads; ++t) s += gW_part[(size_t)t * wsz + x];
        grad_WT[x] = s;
    }
    for (size_t x = 0; x < tsz; ++x) {
        double s = 0.0;
        for (int t = 0; t < nthreads; ++t) s += gT_part[(size_t)t * tsz + x];
        grad_ev_t[x] = s;
    }
    free(gW_part); free(gT_part); free(jobs);
    return 0;
}

/* Per-sample merge of a layer's output spikes into the next layer's sorted
 * event queue (Appendix E.2): order by (time, neuron).  Times are the
 * float32-rounded spike times that the next layer consumes. */
int or_merge(const float* out_t, const int32_t* out_n, int B, int N, int s_max,
             float* ev_t2, int32_t* ev_src2, int32_t* ev_n2, int32_t* perm, int E2_max)
{
    int rc = 0;
    for (int b = 0; b < B; ++b) {
        int cnt = 0;
        for (int i = 0; i < N; ++i) cnt += out_n[(size_t)b * N + i];
        if (cnt > E2_max) { rc = 1; cnt = E2_max; }
        /* Selection of the (time, neuron)-smallest remaining head, one list
         * pointer per neuron: a plain k-way merge. */
        int* head = (int*)calloc((size_t)N, sizeof(int));
        for (int e = 0; e < E2_max; ++e) {
            size_t o = (size_t)b * E2_max + e;
            ev_t2[o] = INFINITY; ev_src2[o] = 0; if (perm) perm[o] = -1;
        }
        for (int e = 0; e < cnt; ++e) {
            int best = -1; float bt = INFINITY;
            for (int i = 0; i < N; ++i) {
                int h = head[i];
                if (h >= out_n[(size_t)b * N + i]) continue;
                float t = out_t[((size_t)b * N + i) * s_max + h];
                if (best < 0 || t < bt) { best = i; bt = t; }
            }
            size_t o = (size_t)b * E2_max + e;
            ev_t2[o] = bt; ev_src2[o] = best;
            if (perm) perm[o] = best * s_max + head[best];
            head[best]++;
        }
        ev_n2[b] = cnt;
        free(head);
    }
    return rc;
}

/* Direct access to the interval rule and the root for the unit pins. */
int or_check_interval(const or_params* p, double V0, double I0, double len, double* hi, double* vmax)
{
    or_check c = check_interval(p, V0, I0, len);
    *hi = c.hi;
    *vmax = c.vmax;
    return c.crossing;
}

double or_solve_root(const or_params* p, double V0, double I0, double hi)
{
    return solve_root(p, V0, I0, hi);
}

/* ---------------------------------------------------------------------- */
/* Learnable synaptic delays (Sec. 3.1 Eq. spike_input; App. E.2 event      */
/* queues).  A spike of input channel j at t_k reaches neuron i at          */
/* a = t_k + d_ij, so every neuron has its own queue: the sample's events   */
/* ordered by arrival.  Readings: the arrival is the float32 sum            */
/* fl(t_k + d_ij) (the same value on every side that builds the queue), and */
/* equal arrivals keep the sample's event order (index k).  The neuron then */
/* runs the serial simulation of simulate_neuron on its queue, with         */
/* out_k counting events of its own queue.  Gradients: the arrival enters   */
/* only through the event's time, so dL/dd_ij sums dL/da over the events of */
/* channel j in neuron i's queue, and dL/dt_k sums dL/da over the neurons.  */
/* ---------------------------------------------------------------------- */

typedef struct { float a; int32_t k; } or_arrival;

static int cmp_arrival(const void* x, const void* y)
{
    const or_arrival* p = (const or_arrival*)x;
    const or_arrival* q = (const or_arrival*)y;
    if (p->a < q->a) return -1;
    if (p->a > q->a) return 1;
    return (p->k > q->k) - (p->k < q->k);
}

/* Neuron i's queue of one sample: arrival times qa[r] and the sample's
 * event index qk[r] of its r-th event, r = 0 .. n - 1. */
static void build_queue(const float* ev_t, const int32_t* ev_src, int n, const float* DT, int N, int i,
                        or_arrival* tmp, float* qa, int32_t* qk, int32_t* qsrc)
{
    for (int k = 0; k < n; ++k) {
        volatile float a = ev_t[k] + DT[(size_t)ev_src[k] * (size_t)N + (size_t)i];
        tmp[k].a = a;
        tmp[k].k = k;
    }
    qsort(tmp, (size_t)n, sizeof(or_arrival), cmp_arrival);
    for (int r = 0; r < n; ++r) {
        qa[r] = tmp[r].a;
        qk[r] = tmp[r].k;
        qsrc[r] = ev_src[tmp[r].k];
    }
}

/* The queues of a batch: q_t, q_k [B][N][E_max] (entries past ev_n[b] are
 * left as they are). */
int or_delay_queues(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                    const float* DT, int C_in, int N, float* q_t, int32_t* q_k)
{
    (void)C_in;
    or_arrival* tmp = (or_arrival*)malloc(sizeof(or_arrival) * (size_t)(E_max > 0 ? E_max : 1));
    int32_t* qs = (int32_t*)malloc(sizeof(int32_t) * (size_t)(E_max > 0 ? E_max : 1));
    if (!tmp || !qs) { free(tmp); free(qs); return -2; }
    for (int b = 0; b < B; ++b)
        for (int i = 0; i < N; ++i) {
            size_t o = ((size_t)b * (size_t)N + (size_t)i) * (size_t)E_max;
            build_queue(ev_t + (size_t)b * E_max, ev_src + (size_t)b * E_max, ev_n[b], DT, N, i, tmp,
                        q_t + o, q_k + o, qs);
        }
    free(tmp); free(qs);
    return 0;
}

typedef struct {
    const or_params* p;
    const float* ev_t; const int32_t* ev_src; const int32_t* ev_n;
    int B, E_max; const float* WT; const float* DT; int C_in, N;
    double* out_t; double* out_i; int32_t* out_k; int32_t* out_n; int32_t* capped; double* tie_t;
    double* min_gap;
    int tid, nthreads;
} dly_fwd_job;

static void* dly_fwd_worker(void* arg)
{
    dly_fwd_job* j = (dly_fwd_job*)arg;
    size_t E = (size_t)(j->E_max > 0 ? j->E_max : 1);
    or_arrival* tmp = (or_arrival*)malloc(sizeof(or_arrival) * E);
    float* qa = (float*)malloc(sizeof(float) * E);
    int32_t* qk = (int32_t*)malloc(sizeof(int32_t) * E);
    int32_t* qs = (int32_t*)malloc(sizeof(int32_t) * E);
    size_t total = (size_t)j->B * (size_t)j->N;
    for (size_t item = (size_t)j->tid; item < total; item += (size_t)j->nthreads) {
        int b = (int)(item / (size_t)j->N), i = (int)(item % (size_t)j->N);
        size_t o = item * (size_t)j->p->s_max;
        for (int s = 0; s < j->p->s_max; ++s) {
            j->out_t[o + s] = INFINITY;
            j->out_i[o + s] = 0.0;
            j->out_k[o + s] = 0;
        }
        int n = j->ev_n[b];
        build_queue(j->ev_t + (size_t)b * j->E_max, j->ev_src + (size_t)b * j->E_max, n, j->DT, j->N, i, tmp,
                    qa, qk, qs);
        or_neuron_result r = simulate_neuron(j->p, qa, qs, n, j->WT, j->N, i, j->out_t + o, j->out_i + o,
                                             j->out_k + o);
        j->out_n[item] = r.n_spikes;
        j->capped[item] = r.capped;
        j->tie_t[item] = r.tie_t;
        j->min_gap[item] = r.min_gap;
    }
    free(tmp); free(qa); free(qk); free(qs);
    return NULL;
}

/* Forward of a layer with delays DT [C_in][N] (d_ij at DT[j*N + i]);
 * outputs as or_forward, out_k counting events of the neuron's queue. */
int or_forward_delayed(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                       const float* WT, const float* DT, int C_in, int N, const or_params* p, int nthreads,
                       double* out_t, double* out_i, int32_t* out_k, int32_t* out_n, int32_t* capped,
                       double* tie_t, double* min_gap)
{
    if (!(p->tau_mem > p->tau_syn && p->tau_syn > 0.0) || !(p->v_reset < p->v_th) || p->s_max < 1)
        return -1;
    if (nthreads < 1) nthreads = 1;
    dly_fwd_job* jobs = (dly_fwd_job*)calloc((size_t)nthreads, sizeof(dly_fwd_job));
    if (!jobs) return -2;
    for (int t = 0; t < nthreads; ++t) {
        dly_fwd_job j = {p, ev_t, ev_src, ev_n, B, E_max, WT, DT, C_in, N,
                         out_t, out_i, out_k, out_n, capped, tie_t, min_gap, t, nthreads};
        jobs[t] = j;
    }
    int rc = run_threads(dly_fwd_worker, jobs, sizeof(dly_fwd_job), nthreads);
    free(jobs);
    return rc;
}

typedef struct {
    const or_params* p;
    const float* ev_t; const int32_t* ev_src; const int32_t* ev_n;
    int B, E_max; const float* WT; const float* DT; int C_in, N;
    const double* out_t; const double* out_i; const int32_t* out_k; const int32_t* out_n;
    const double* grad_out_t;
    double* gW_part;   /* [nthreads][C_in][N] */
    double* gD_part;   /* [nthreads][C_in][N] */
    double* gT_part;   /* [nthreads][B][E_max] */
    int tid, nthreads;
} dly_bwd_job;

static void* dly_bwd_worker(void* arg)
{
    dly_bwd_job* j = (dly_bwd_job*)arg;
    const or_params* p = j->p;
    const double tm = p->tau_mem, ts = p->tau_syn, ka = kappa(p);
    const int smax = p->s_max;
    size_t E = (size_t)(j->E_max > 0 ? j->E_max : 1);
    double* mu = (double*)malloc(sizeof(double) * (size_t)smax);
    or_arrival* tmp = (or_arrival*)malloc(sizeof(or_arrival) * E);
    float* qa = (float*)malloc(sizeof(float) * E);
    int32_t* qk = (int32_t*)malloc(sizeof(int32_t) * E);
    int32_t* qs = (int32_t*)malloc(sizeof(int32_t) * E);
    size_t wsz = (size_t)j->C_in * (size_t)j->N;
    double* gW = j->gW_part + (size_t)j->tid * wsz;
    double* gD = j->gD_part + (size_t)j->tid * wsz;
    double* gT = j->gT_part + (size_t)j->tid * (size_t)j->B * (size_t)j->E_max;
    size_t total = (size_t)j->B * (size_t)j->N;
    for (size_t item = (size_t)j->tid; item < total; item += (size_t)j->nthreads) {
        int b = (int)(item / (size_t)j->N), i = (int)(item % (size_t)j->N);
        int ns = j->out_n[item];
        if (ns <= 0) continue;
        const double* ts_ = j->out_t + item * (size_t)smax;
        const double* is_ = j->out_i + item * (size_t)smax;
        const int32_t* ks_ = j->out_k + item * (size_t)smax;
        const double* g = j->grad_out_t + item * (size_t)smax;
        /* the adjoints of the spikes, as in bwd_worker */
        for (int s = ns - 1; s >= 0; --s) {
            double lam = g[s];
            for (int s2 = s + 1; s2 < ns; ++s2)
                lam -= (p->v_th - p->v_reset) / tm * mu[s2] * exp(-(ts_[s2] - ts_[s]) / tm);
            double vp = dvdt(p, p->v_th, is_[s]);
            if (vp < p->solver_reg) vp = p->solver_reg;
            mu[s] = -lam / vp;
        }
        int n = j->ev_n[b];
        build_queue(j->ev_t + (size_t)b * j->E_max, j->ev_src + (size_t)b * j->E_max, n, j->DT, j->N, i, tmp,
                    qa, qk, qs);
        /* each queue event before a spike: dF_s/dw = K(t_s - a_r),
         * dF_s/da_r = -w K'(t_s - a_r) */
        for (int r = 0; r < n; ++r) {
            if (r >= ks_[ns - 1]) break;
            double ar = (double)qa[r];
            double a = 0.0, ad = 0.0;
            for (int s = 0; s < ns; ++s) {
                if (r >= ks_[s]) continue;
                double u = ts_[s] - ar;
                if (u < 0.0) u = 0.0;
                double em = exp(-u / tm), es2 = exp(-u / ts);
                a += mu[s] * ka * (em - es2);
                ad += mu[s] * ka * (-em / tm + es2 / ts);
            }
            size_t wi = (size_t)qs[r] * (size_t)j->N + (size_t)i;
            double w = (double)j->WT[wi];
            gW[wi] += a;
            gD[wi] += -w * ad;
            gT[(size_t)b * j->E_max + qk[r]] += -w * ad;
        }
    }
    free(mu); free(tmp); free(qa); free(qk); free(qs);
    return NULL;
}

/* Backward of a layer with delays: grad_WT, grad_DT [C_in][N] and
 * grad_ev_t [B][E_max] overwritten, from the delayed forward's outputs. */
int or_backward_delayed(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                        const float* WT, const float* DT, int C_in, int N, const or_params* p, int nthreads,
                        const double* out_t, const double* out_i, const int32_t* out_k, const int32_t* out_n,
                        const double* grad_out_t, double* grad_WT, double* grad_DT, double* grad_ev_t)
{
    if (nthreads < 1) nthreads = 1;
    size_t wsz = (size_t)C_in * (size_t)N, tsz = (size_t)B * (size_t)E_max;
    double* gW_part = (double*)calloc(wsz * (size_t)nthreads, sizeof(double));
    double* gD_part = (double*)calloc(wsz * (size_t)nthreads, sizeof(double));
    double* gT_part = (double*)calloc(tsz * (size_t)nthreads + 1, sizeof(double));
    dly_bwd_job* jobs = (dly_bwd_job*)calloc((size_t)nthreads, sizeof(dly_bwd_job));
    if (!gW_part || !gD_part || !gT_part || !jobs) {
        free(gW_part); free(gD_part); free(gT_part); free(jobs);
        return -2;
    }
    for (int t = 0; t < nthreads; ++t) {
        dly_bwd_job j = {p, ev_t, ev_src, ev_n, B, E_max, WT, DT, C_in, N, out_t, out_i, out_k, out_n, grad_out_t,
                         gW_part, gD_part, gT_part, t, nthreads};
        jobs[t] = j;
    }
    run_threads(dly_bwd_worker, jobs, sizeof(dly_bwd_job), nthreads);
    for (size_t x = 0; x < wsz; ++x) {
        double s = 0.0, sd = 0.0;
        for (int t = 0; t < nthreads; ++t) {
            s += gW_part[(size_t)t * wsz + x];
            sd += gD_part[(size_t)t * wsz + x];
        }
        grad_WT[x] = s;
        grad_DT[x] = sd;
    }
    for (size_t x = 0; x < tsz; ++x) {
        double s = 0.0;
        for (int t = 0; t < nthreads; ++t) s += gT_part[(size_t)t * tsz + x];
        grad_ev_t[x] = s;
    }
    free(gW_part); free(gD_part); free(gT_part); free(jobs);
    return 0;
}
