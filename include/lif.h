/*
 * lif.h -- C ABI of the MI355X (gfx950) event-driven LIF layer library
 * (liblif.so), after "Bullet Trains: Parallelizing Training of Temporally
 * Precise Spiking Neural Networks" (arXiv 2603.13283).
 *
 * Conventions shared by every entry point
 *   - Array arguments are DEVICE pointers unless stated otherwise; the caller
 *     allocates and owns every buffer (outputs and workspace included).  The
 *     library never allocates device memory, never synchronises the stream
 *     and keeps no state between calls (except the optional kernel timer,
 *     see lif_timer_*, and the fixed workspace array of
 *     lif_layer_forward_noalloc).  Every behaviour is set by the arguments
 *     (no environment variables are read).
 *   - Work is enqueued on `stream` (a hipStream_t; NULL is the null stream)
 *     and the call returns at once.  Calls on different streams with
 *     distinct buffers may run concurrently.
 *   - Argument errors are detected on the host before anything is launched;
 *     the call then returns a negative LIF_ERR_* code and enqueues nothing.
 *     Conditions that depend on the data (spike cap reached, unsorted input
 *     under LIF_VALIDATE, merge overflow) are reported in the device status
 *     words (int32[LIF_STATUS_WORDS]), which the call resets itself.
 *     Malformed queues never make a kernel address outside its buffers:
 *     event counts are clamped into [0, E_max] and sources into [0, C_in).
 *   - Times are in seconds relative to the sample start t = 0, where every
 *     neuron is at rest (V = I = 0).  Index layouts are row-major.
 *   - Input events of one sample are sorted by time (ties in any order);
 *     entries k >= ev_n[b] are padding and are never read as events.
 *
 * Model (paper Sec. 3.1, Appendix A): tau_m dV/dt = -V + I,
 * tau_s dI/dt = -I; an input event from channel c adds w_{i c} to I of
 * neuron i (Eq. spike_input, no delays); neuron i emits a spike when
 * V >= V_th and V is then hard-reset to V_reset (I is not reset).
 */
#ifndef LIF_H
#define LIF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Same type as hipStream_t. */
typedef struct ihipStream_t* lif_stream_t;

/* Return codes. */
#define LIF_OK              0
#define LIF_ERR_ARG        -1  /* null pointer, bad size, s_max < 1          */
#define LIF_ERR_TAU        -2  /* require tau_mem > tau_syn > 0 (App. D.1)   */
#define LIF_ERR_THRESHOLD  -3  /* require 0 < v_th and v_reset < v_th        */
#define LIF_ERR_WORKSPACE  -4  /* ws_bytes below the *_workspace_size value  */
#define LIF_ERR_HIP        -5  /* a kernel launch failed                     */
#define LIF_ERR_SIZE       -6  /* a size exceeds a documented limit          */
/* Size limits: C_in * N_out < 2^29 (W^T is addressed with 32-bit byte
   offsets); B * E_max < 2^40. */

/* lif_params.flags */
#define LIF_VALIDATE      1u  /* check sorted times, finite values, source range */
#define LIF_ROOT_GENERAL  2u  /* solve spike times with the exponential Newton
                                 iteration even when tau_m / tau_s is an integer
                                 plus one (where a polynomial solve is used by
                                 default); both give the same spike times to
                                 float64 rounding.  For tests of that path.    */

/* Device status words written by every forward call (int32 each). */
#define LIF_STATUS_WORDS     8
#define LIF_ST_FLAGS         0  /* OR of LIF_WARN_* bits                     */
#define LIF_ST_CAPPED        1  /* neurons that reached s_max spikes         */
#define LIF_ST_SPIKES        2  /* output spikes emitted                     */
#define LIF_ST_CAND_BLOCKS   3  /* event sub-blocks flagged by the scan      */
#define LIF_ST_WALKED_BLOCKS 4  /* flagged sub-blocks handed to the resolve
                                   pass (equal to LIF_ST_CAND_BLOCKS)       */
#define LIF_ST_ROOT_SOLVES   5  /* spike-time root solves                    */
#define LIF_ST_EVENTS        6  /* input events consumed (sum of ev_n)       */
#define LIF_ST_POOL_FALLBACK 7  /* flagged sub-blocks past the pool's
                                   capacity (rebuilt by a slower re-walk)   */

#define LIF_WARN_SPIKE_CAP   1  /* a neuron stopped at s_max spikes          */
#define LIF_WARN_UNSORTED    2  /* LIF_VALIDATE: times decrease in a sample  */
#define LIF_WARN_BAD_SOURCE  4  /* LIF_VALIDATE: source outside [0, C_in)    */
#define LIF_WARN_NONFINITE   8  /* LIF_VALIDATE: NaN/inf event time          */
#define LIF_WARN_MERGE_FULL 16  /* merge: more spikes than E2_max            */
#define LIF_WARN_BAD_COUNT  32  /* LIF_VALIDATE: ev_n[b] outside [0, E_max]  */
#define LIF_WARN_INTERNAL   64  /* internal error: a cross-workgroup wait gave
                                   up (results are not valid)                */
#define LIF_WARN_BAD_DELAY 128  /* lif_delay_queues: a delay is negative or
                                   not finite (queue order unspecified)      */

typedef struct lif_params {
    double   tau_mem;    /* tau_m (s); must exceed tau_syn (paper: 0.02)        */
    double   tau_syn;    /* tau_s (s); > 0 (paper: 0.005)                       */
    double   v_th;       /* threshold V_th > 0, above rest (paper: 1.0)         */
    double   v_reset;    /* reset potential, < v_th (paper: 0.0)                */
    double   t_end;      /* end of the interval after the last event; +INFINITY
                            (events later than t_end are still consumed; the
                            open interval is then empty)                        */
    int32_t  s_max;      /* output spike capacity per neuron, >= 1 (App. E.2)   */
    uint32_t flags;      /* LIF_VALIDATE, LIF_ROOT_GENERAL                      */
    double   solver_reg; /* backward floor on dV/dt at a spike (paper 0.01,
                            App. E hyperparameter table, "Solver
                            Regularization"); 0 disables it                     */
    int32_t  pool_cap;   /* forward: pool entries per sample (16 bytes each,
                            the entering state of a flagged event block);
                            < 0 selects the library's default.  Blocks past
                            the entries are rebuilt by a slower path with
                            identical results (0: every block is; for tests
                            of that path).  Enters the workspace size.        */
    int32_t  reserved;   /* must be 0                                           */
} lif_params;

/* Library version string (static storage). */
const char* lif_version(void);

/* --------------------------------------------------------------------- */
/* Forward pass of one layer (paper Sec. 3.2.1 parallel scan of the affine  */
/* event maps, Eq. affine and the Combine operator; Sec. 3.2.2 interval    */
/* rule with t_Vmax of Eq. t_vmax; Appendix D.1 Newton spike-time solve;   */
/* Appendix E.2 single commit + restart after each spike).                 */
/*                                                                         */
/*   ev_t   float [B][E_max]   event times, sorted per sample              */
/*   ev_src int32 [B][E_max]   source channel of each event, in [0, C_in)  */
/*   ev_n   int32 [B]          events per sample, 0 <= ev_n[b] <= E_max    */
/*   WT     float [C_in][N_out] weights, WT[c*N_out + i] = w_{i c}         */
/*   out_t  float [B][N_out][s_max] spike times in increasing order,       */
/*                             +INFINITY after the last spike              */
/*   out_n  int32 [B][N_out]   spike counts                                */
/*   out_i  float [B][N_out][s_max] synaptic current I at each spike (the  */
/*                             backward pass needs it); 0 padding; may be  */
/*                             NULL                                        */
/*   out_k  int32 [B][N_out][s_max] input events consumed before each      */
/*                             spike: the spike lies in the interval that  */
/*                             event out_k closes (or after the last event */
/*                             when out_k = ev_n[b]), and depends on       */
/*                             events 0 .. out_k - 1 only; 0 padding; the  */
/*                             backward pass needs it; may be NULL         */
/*   status int32 [LIF_STATUS_WORDS]                                       */
/*   ws     device workspace of ws_bytes >= lif_layer_forward_workspace_size */
/* The spike times are exact up to float64 rounding of the closed-form     */
/* dynamics and are returned rounded to float32.                           */
/* --------------------------------------------------------------------- */
size_t lif_layer_forward_workspace_size(int B, int E_max, int C_in, int N_out, const lif_params* p);

int lif_layer_forward(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                      const float* WT, int C_in, int N_out, const lif_params* p,
                      float* out_t, int32_t* out_n, float* out_i, int32_t* out_k, int32_t* status,
                      void* ws, size_t ws_bytes, lif_stream_t stream);

/* The sequential baseline (paper Appendix E.3): one GPU thread per
 * (sample, neuron) consumes every event in order and runs the same interval
 * rule and root solve.  Same arguments and results as lif_layer_forward;
 * its workspace size is lif_layer_forward_workspace_size as well. */
int lif_layer_forward_sequential(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B,
                                 int E_max, const float* WT, int C_in, int N_out, const lif_params* p,
                                 float* out_t, int32_t* out_n, float* out_i, int32_t* out_k,
                                 int32_t* status, void* ws, size_t ws_bytes, lif_stream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * forward pass of lif_layer_forward, with the same arguments and results
 * but no ws/ws_bytes.  Its workspace is a fixed array of
 * lif_layer_forward_noalloc_max_bytes() bytes (64 MiB) in each GPU's
 * memory, held from the library's load until the process ends; the call
 * allocates nothing.  The default pool (pool_cap < 0) is cut to what the
 * array holds (the blocks past it take the rebuild path: results are
 * unchanged); LIF_ERR_SIZE when the layout without pool entries, or with a
 * pool_cap the caller set, exceeds the array.  LIF_ERR_HIP when the array's
 * device address cannot be obtained.  Every call on a GPU uses that GPU's
 * one array: calls that overlap on one GPU (different streams, or several
 * host threads) race, and the caller must order them. */
int lif_layer_forward_noalloc(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                              const float* WT, int C_in, int N_out, const lif_params* p,
                              float* out_t, int32_t* out_n, float* out_i, int32_t* out_k, int32_t* status,
                              lif_stream_t stream);
size_t lif_layer_forward_noalloc_max_bytes(void);

/* The paper's own chunked scheme, for studies of the chunk size and the
 * work retained (Sec. 3.2.1 "Speculative execution" and "Fixed compute
 * budget", Appendix E.2, Appendix G): one wave per (sample, neuron) takes
 * its queue K events at a time (K = 64, 128 or 256), scans the chunk's
 * affine maps across the wave, tests every interval with the rule of
 * Sec. 3.2.2 and commits only the first crossing (bracket of Appendix D.2,
 * multisection to the smallest double with V >= V_th); the next iteration
 * restarts at the spike with the same pending event.  At most C iterations
 * run per neuron (C <= 0: ceil(E_max / K) + s_max, the paper's budget for
 * an input layer) and at most s_max spikes are kept.  Outputs as
 * lif_layer_forward (out_k included), and per (sample, neuron):
 *   consumed  int32 [B][N_out] input events consumed when the neuron stopped
 *   processed int32 [B][N_out] input events of all its chunk iterations (an
 *             event visited twice counts twice); may be NULL, as consumed
 * Status words: LIF_ST_CAND_BLOCKS counts chunk iterations and
 * LIF_ST_WALKED_BLOCKS processed events; the others as the forward.
 * With a budget that suffices, the spikes are those of lif_layer_forward.
 * No workspace. */
int lif_layer_forward_chunked(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                              const float* WT, int C_in, int N_out, const lif_params* p, int K, int C,
                              float* out_t, int32_t* out_n, float* out_i, int32_t* out_k, int32_t* consumed,
                              int32_t* processed, int32_t* status, lif_stream_t stream);

/* A layer with learnable synaptic delays (Sec. 3.1 Eq. spike_input: a spike
 * of input channel j at t_k reaches neuron i at t_k + d_ij; Appendix E.2:
 * a sorted event queue per neuron).  Three calls: the queues, then the
 * forward and the backward on them.
 *
 * lif_delay_queues: neuron i's queue of sample b lists the sample's events
 * ordered by (arrival, k), with the arrival the float32 sum
 * a = t_k + DT[src_k * N_out + i] (DT: delays d_ij >= 0 in seconds, W^T
 * layout [C_in][N_out]).
 *   q_t  float [B][N_out][E_max]  arrival time of each queue entry
 *   q_k  int32 [B][N_out][E_max]  the sample's event index of each entry
 * Entries past ev_n[b] are not written.  status (nullable) int32
 * [LIF_STATUS_WORDS]: reset, then LIF_ST_EVENTS and LIF_WARN_BAD_DELAY in
 * LIF_ST_FLAGS when some delay is negative or not finite (the queues are
 * then in bounds, their order unspecified).  ws: at least
 * lif_delay_queues_workspace_size(B, E_max, N_out) bytes (4 per queue entry, 12
 * when E_max > 16384).
 * Errors: LIF_ERR_ARG, LIF_ERR_SIZE (B * N_out >= 2^31 or B > 65535),
 * LIF_ERR_WORKSPACE. */
size_t lif_delay_queues_workspace_size(int B, int E_max, int N_out);
int lif_delay_queues(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                     const float* DT, int C_in, int N_out, float* q_t, int32_t* q_k, int32_t* status,
                     void* ws, size_t ws_bytes, lif_stream_t stream);

/* Forward of the delayed layer on the queues of lif_delay_queues (the
 * sample's ev_src/ev_n with them): every neuron runs the interval rule and
 * spike solve of the layer on its own queue (the chunked walk of
 * lif_layer_forward_chunked with K = 128 and no budget: the queue is
 * consumed unless the neuron stops at s_max).  Outputs as
 * lif_layer_forward; out_k counts events of the neuron's own queue.  Status
 * words as lif_layer_forward_chunked.  No workspace. */
int lif_layer_forward_delayed(const float* q_t, const int32_t* q_k, const int32_t* ev_src, const int32_t* ev_n,
                              int B, int E_max, const float* WT, int C_in, int N_out, const lif_params* p,
                              float* out_t, int32_t* out_n, float* out_i, int32_t* out_k, int32_t* status,
                              lif_stream_t stream);

/* The sequential baseline of the delayed layer (Appendix E.3): one thread
 * per (sample, neuron) takes its queue one event at a time with the same
 * interval rule and spike solve.  Same arguments and outputs as
 * lif_layer_forward_delayed; status words as lif_layer_forward_sequential. */
int lif_layer_forward_delayed_sequential(const float* q_t, const int32_t* q_k, const int32_t* ev_src,
                                         const int32_t* ev_n, int B, int E_max, const float* WT, int C_in,
                                         int N_out, const lif_params* p, float* out_t, int32_t* out_n,
                                         float* out_i, int32_t* out_k, int32_t* status, lif_stream_t stream);

/* Backward of the delayed layer (Appendix D.3 on each neuron's queue): for
 * L = sum grad_out_t * out_t, from the delayed forward's outputs,
 *   grad_WT    float [C_in][N_out]  dL/dw_ij, overwritten
 *   grad_DT    float [C_in][N_out]  dL/dd_ij, overwritten (nullable)
 *   grad_ev_t  float [B][E_max]     dL/dt_k summed over the neurons,
 *                                   overwritten (nullable; 0 past ev_n[b])
 * Bitwise reproducible (64-bit fixed-point sums).  ws: at least
 * lif_layer_backward_delayed_workspace_size(...) bytes, which include 8
 * bytes per (sample, neuron, queue event) for the dL/dt terms: with
 * grad_ev_t NULL, B * N_out * E_max * 8 bytes less suffice.  Errors as
 * lif_layer_backward. */
size_t lif_layer_backward_delayed_workspace_size(int B, int E_max, int C_in, int N_out, const lif_params* p);
int lif_layer_backward_delayed(const float* q_t, const int32_t* q_k, const int32_t* ev_src, const int32_t* ev_n,
                               int B, int E_max, const float* WT, int C_in, int N_out, const lif_params* p,
                               const float* out_t, const int32_t* out_n, const float* out_i,
                               const int32_t* out_k, const float* grad_out_t, float* grad_WT, float* grad_DT,
                               float* grad_ev_t, void* ws, size_t ws_bytes, lif_stream_t stream);

/* --------------------------------------------------------------------- */
/* Backward pass (paper Appendix D.3, Eq. ift_vjp, chained through the     */
/* hard resets): given dL/dt for every output spike, returns dL/dW and     */
/* dL/d(event time).                                                       */
/*                                                                         */
/*   out_t, out_n, out_i, out_k  the forward results for the same inputs */
/*                        (out_i and out_k are required here)              */
/*   grad_out_t float [B][N_out][s_max]  dL/dt_s; padding entries ignored  */
/*   grad_WT    float [C_in][N_out]      overwritten with dL/dWT           */
/*   grad_ev_t  float [B][E_max]         overwritten with dL/dev_t (0 on   */
/*                                       padding); may be NULL             */
/* dV/dt at each spike is floored at p->solver_reg.  Which input events a  */
/* spike depends on is read from out_k, not from comparing the (float32)   */
/* times, so an event that the rounding of a spike time puts at the same   */
/* time still counts as before it.  grad_WT sums over samples with float64 */
/* atomics, so its last bits can depend on timing.                         */
/* --------------------------------------------------------------------- */
size_t lif_layer_backward_workspace_size(int B, int E_max, int C_in, int N_out, const lif_params* p);

int lif_layer_backward(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                       const float* WT, int C_in, int N_out, const lif_params* p,
                       const float* out_t, const int32_t* out_n, const float* out_i, const int32_t* out_k,
                       const float* grad_out_t, float* grad_WT, float* grad_ev_t,
                       void* ws, size_t ws_bytes, lif_stream_t stream);

/* --------------------------------------------------------------------- */
/* Layer merge (paper Appendix E.2): the spikes of a layer become the next */
/* layer's sorted per-sample event queue, ordered by (time, neuron).       */
/*                                                                         */
/*   out_t, out_n   a forward result, [B][N][s_max] and [B][N]             */
/*   ev_t2   float [B][E2_max]  merged times (+INFINITY padding)           */
/*   ev_src2 int32 [B][E2_max]  source = emitting neuron index             */
/*   ev_n2   int32 [B]          merged counts (clipped at E2_max: a sample */
/*                              with more spikes keeps its E2_max earliest  */
/*                              in (time, neuron) order)                    */
/*   perm    int32 [B][E2_max]  i*s_max + s of each merged spike, -1 on    */
/*                              padding; may be NULL                       */
/*   status  int32 [LIF_STATUS_WORDS] (LIF_WARN_MERGE_FULL on overflow)    */
/* Limit: E2_max <= LIF_MERGE_MAX (LIF_ERR_SIZE otherwise).                */
/* --------------------------------------------------------------------- */
#define LIF_MERGE_MAX 16384
size_t lif_merge_workspace_size(int B, int N, int s_max, int E2_max);

int lif_merge_spikes(const float* out_t, const int32_t* out_n, int B, int N, int s_max,
                     float* ev_t2, int32_t* ev_src2, int32_t* ev_n2, int32_t* perm, int E2_max,
                     int32_t* status, void* ws, size_t ws_bytes, lif_stream_t stream);

/* --------------------------------------------------------------------- */
/* First-spike readout loss: logits_c = -t_c / tau0 from the first spike   */
/* time t_c of readout neuron c (t_silent when it never fires), mean       */
/* softmax cross-entropy over the batch, and dL/dt written into the s = 0  */
/* slot of grad_out_t (all other slots and silent neurons get 0).          */
/*   labels int32 [B] in [0, N); loss float [1] (device)                   */
/* --------------------------------------------------------------------- */
int lif_first_spike_ce(const float* out_t, const int32_t* out_n, int B, int N, int s_max,
                       const int32_t* labels, double tau0, double t_silent,
                       float* loss, float* grad_out_t, lif_stream_t stream);

/* --------------------------------------------------------------------- */
/* Gradient of a merged queue's event times back to the spikes it was      */
/* made of (the inverse of lif_merge_spikes' permutation): grad_out_t      */
/* [B][N][s_max] gets grad_ev_t2[b][j] in slot perm[b][j] for the queue's  */
/* events j < ev_n2[b], and 0 in every other slot.                         */
/* --------------------------------------------------------------------- */
int lif_merge_grad(const float* grad_ev_t2, const int32_t* perm, const int32_t* ev_n2, int B, int E2_max,
                   int N, int s_max, float* grad_out_t, lif_stream_t stream);

/* --------------------------------------------------------------------- */
/* The paper's readout and classification loss (Sec. 3.3, Appendix C):    */
/* one leaky integrator (LI) per class, with the LIF neuron's V/I dynamics */
/* (Eq. mem_pot) and no spikes, fed by the last hidden layer's merged      */
/* queue with weights W^T [C_in][N_cls]; its logit is                      */
/*   z_c = integral over [0, tau_max] of e^{-t/tau_li} V_c(t) dt           */
/* (Eq. weighted_leaky_integrator_full; tau_li = +INFINITY gives the       */
/* unweighted integral of Eq. leaky_integrator), and the loss is the mean  */
/* softmax cross-entropy of beta z (the fixed temperature multiplier of    */
/* Appendix C).  Events at or after tau_max add nothing.                   */
/*   logits    float [B][N_cls] z before the temperature; may be NULL      */
/*   labels    int32 [B] in [0, N_cls) (clamped); NULL: logits only       */
/*   loss      float [1] device; may be NULL                               */
/*   grad_WT   float [C_in][N_cls] dL/dW^T, overwritten; may be NULL       */
/*   grad_ev_t float [B][E_max] dL/d(event time), 0 on padding; may be     */
/*             NULL (route it to the spikes with lif_merge_grad)           */
/* Sums run in a fixed order (no floating-point atomics): results are      */
/* bitwise reproducible.  Limit: N_cls <= LIF_LI_MAX_CLASSES.              */
/* --------------------------------------------------------------------- */
#define LIF_LI_MAX_CLASSES 64
typedef struct lif_li_params {
    double tau_mem;     /* tau_m of the LI neurons (s), > tau_syn            */
    double tau_syn;     /* tau_s (s), > 0                                    */
    double tau_li;      /* weighting time constant (s), > 0; +INFINITY: none */
    double tau_max;     /* end of the integration window (s), > 0            */
    double beta;        /* logit temperature multiplier                      */
} lif_li_params;

size_t lif_li_readout_workspace_size(int B, int E_max, int C_in, int N_cls);

int lif_li_readout(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                   const float* WT, int C_in, int N_cls, const lif_li_params* q, const int32_t* labels,
                   float* logits, float* loss, float* grad_WT, float* grad_ev_t, void* ws, size_t ws_bytes,
                   lif_stream_t stream);

/* --------------------------------------------------------------------- */
/* Spike-count regularisers (Appendix E.1, Eq. loss) of a layer, from its  */
/* inputs and the forward's spikes.  For each (sample b, neuron i) and     */
/* each input interval j (between events j - 1 and j, t_{-1} = 0, and the  */
/* open interval after the last event up to t_end), V_max is the largest  */
/* V of the interval's trajectory from its true start state (the resets of */
/* earlier intervals applied, none inside it); interval j is spiking when  */
/* a spike has out_k = j, else silent.                                     */
/*   under[b][i] = mean over silent intervals of max(V_th - V_max, 0)       */
/*   over[b][i]  = mean over spiking intervals of max(V_max - V_th, 0)      */
/* (0 for an empty set), and with c = spike counts (out_n), the gates      */
/* g_u = max(1 - mean_b c / c_target, 0), g_o = max(mean_b c / c_target - 1, 0): */
/*   loss[0] = L_reg  = mean_i (g_u mean_b under + g_o mean_b over)         */
/*   loss[1] = L_over = (1/N) sum_i sum_b max(c / c_target - 1, 0) over     */
/* The caller weights them (lambda_reg, lambda_over-reg of Eq. loss).      */
/*   under, over  float [B][N_out]; may be NULL                            */
/* Sums run in a fixed order: results are bitwise reproducible.            */
/* --------------------------------------------------------------------- */
size_t lif_spike_count_reg_workspace_size(int B, int E_max, int C_in, int N_out);

int lif_spike_count_reg(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                        const float* WT, int C_in, int N_out, const lif_params* p, const float* out_t,
                        const int32_t* out_n, const int32_t* out_k, double c_target, float* loss, float* under,
                        float* over, void* ws, size_t ws_bytes, lif_stream_t stream);

/* Gradient of lambda_reg L_reg + lambda_over L_over (the loss values of
 * lif_spike_count_reg, also written to loss[2] when loss is not NULL), the
 * gates held constant (they are functions of the spike counts).  Each V_max
 * is the interval trajectory's value at its argmax, which depends on the
 * weights and input times before the interval, on the spike times before it
 * (through the resets), and, when the argmax is an interval end that is an
 * input time, on that time.  Outputs:
 *   grad_spike float [B][N_out][s_max]  the upstream gradient on the layer's
 *              spike times, ADDED to what the array holds: run
 *              lif_layer_backward with it (together with the downstream
 *              loss's spike-time gradient) for the part through the spikes
 *   grad_WT    float [C_in][N_out]      the direct part of dL/dW, overwritten
 *   grad_ev_t  float [B][E_max]         the direct part of dL/dt_in,
 *              overwritten (nullable; 0 past ev_n[b])
 * The full gradient is the direct part plus that backward pass.  Bitwise
 * reproducible.  ws: lif_spike_count_reg_backward_workspace_size(...) bytes
 * (about 16 bytes per (sample, interval, neuron)).  Errors as
 * lif_spike_count_reg, LIF_ERR_ARG also for a non-finite lambda. */
size_t lif_spike_count_reg_backward_workspace_size(int B, int E_max, int C_in, int N_out);

int lif_spike_count_reg_backward(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                                 const float* WT, int C_in, int N_out, const lif_params* p, const float* out_t,
                                 const int32_t* out_n, const int32_t* out_k, double c_target, double lam_reg,
                                 double lam_over, float* loss, float* grad_spike, float* grad_WT, float* grad_ev_t,
                                 void* ws, size_t ws_bytes, lif_stream_t stream);

/* Spike-count regularisers of a layer with synaptic delays: the same terms */
/* as lif_spike_count_reg with each neuron's intervals lying between        */
/* consecutive arrivals of its own queue (Sec. 3.1 Eq. spike_input, App.    */
/* E.2): interval r of neuron i ends at its queue event r, interval ev_n[b] */
/* is the open one up to t_end, and a spike belongs to interval out_k (the  */
/* queue events consumed before it, as lif_layer_forward_delayed counts).   */
/*   q_t, q_k   the queues of lif_delay_queues ([B][N_out][E_max])          */
/*   out_*      lif_layer_forward_delayed's outputs for them                */
/*   loss, under, over  as lif_spike_count_reg (all nullable)               */
/* ws: lif_spike_count_reg_delayed_workspace_size(...) bytes (the same size */
/* serves the backward below).  Bitwise reproducible.  Errors as            */
/* lif_spike_count_reg.                                                     */
/* Backward: the gradient of lambda_reg L_reg + lambda_over L_over with the */
/* gates held constant, an arrival's term going to both its input time and  */
/* its delay (d a / d t = d a / d d = 1):                                   */
/*   grad_spike float [B][N_out][s_max]  ADDED to (run                      */
/*              lif_layer_backward_delayed with it for the part through     */
/*              the spikes)                                                 */
/*   grad_WT, grad_DT float [C_in][N_out], grad_ev_t float [B][E_max]: the  */
/*              direct parts, overwritten (grad_DT, grad_ev_t nullable)     */
/* about 8 bytes per (sample, neuron, queue event) of workspace.            */
/* --------------------------------------------------------------------- */
size_t lif_spike_count_reg_delayed_workspace_size(int B, int E_max, int C_in, int N_out);

int lif_spike_count_reg_delayed(const float* q_t, const int32_t* q_k, const int32_t* ev_src, const int32_t* ev_n,
                                int B, int E_max, const float* WT, int C_in, int N_out, const lif_params* p,
                                const float* out_t, const int32_t* out_n, const int32_t* out_k, double c_target,
                                float* loss, float* under, float* over, void* ws, size_t ws_bytes,
                                lif_stream_t stream);

int lif_spike_count_reg_delayed_backward(const float* q_t, const int32_t* q_k, const int32_t* ev_src,
                                         const int32_t* ev_n, int B, int E_max, const float* WT, int C_in,
                                         int N_out, const lif_params* p, const float* out_t, const int32_t* out_n,
                                         const int32_t* out_k, double c_target, double lam_reg, double lam_over,
                                         float* loss, float* grad_spike, float* grad_WT, float* grad_DT,
                                         float* grad_ev_t, void* ws, size_t ws_bytes, lif_stream_t stream);

/* --------------------------------------------------------------------- */
/* Adam step (the optimiser the paper trains with, App. E): for each of    */
/* the n parameters, m1 = b1 m1 + (1 - b1) g, m2 = b2 m2 + (1 - b2) g^2,   */
/* p -= lr (m1 / (1 - b1^step)) / (sqrt(m2 / (1 - b2^step)) + eps), in     */
/* float64, stored in float32.  step >= 1 counts the updates so far.       */
/* param, m1, m2 are updated in place; the moments start at 0.            */
/* --------------------------------------------------------------------- */
typedef struct lif_adam_params {
    double lr, beta1, beta2, eps;
} lif_adam_params;

int lif_adam_step(float* param, const float* grad, float* m1, float* m2, size_t n, const lif_adam_params* a,
                  int step, lif_stream_t stream);

/* Elementwise pieces of the training step.  lif_add: y[i] += x[i] (adds the
 * direct part of a regulariser gradient to a layer's gradient).
 * lif_softplus: d[i] = log(1 + e^{beta x[i]}) / beta, the delay activation
 * of App. E.5 (beta = the softplus sharpness, > 0); lif_softplus_grad:
 * grad_x[i] = grad_d[i] sigmoid(beta x[i]).  Computed in float64, stored in
 * float32; LIF_ERR_ARG on a null pointer with n > 0 or beta <= 0. */
int lif_add(float* y, const float* x, size_t n, lif_stream_t stream);
int lif_softplus(const float* x, float* d, size_t n, double beta, lif_stream_t stream);
int lif_softplus_grad(const float* x, const float* grad_d, float* grad_x, size_t n, double beta,
                      lif_stream_t stream);

/* --------------------------------------------------------------------- */
/* Optional kernel timer (host-side state, off by default).  When enabled, */
/* every kernel launched by this library is launched with a pair of HIP    */
/* events that its own dispatch records (hipExtLaunchKernel), so each      */
/* elapsed time is the kernel's execution on its stream; lif_timer_read    */
/* synchronises on the recorded events and returns per-kernel totals.      */
/*   lif_timer_enable(1) resets and starts recording, (0) stops.           */
/*   lif_timer_read fills up to `cap` entries: names[j] (static strings),  */
/*   total_ms[j], launches[j]; returns the number of kernels seen.         */
/* --------------------------------------------------------------------- */
void lif_timer_enable(int on);
int lif_timer_read(const char** names, double* total_ms, int32_t* launches, int cap);

#ifdef __cplusplus
}
#endif

#endif /* LIF_H */
