// lif_host.hpp -- host-side helpers shared by the library's entry points:
// argument validation, model constants, workspace layout, launch timing.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#include "../../include/lif.h"
#include "lif_common.hpp"

namespace lif {

struct FwdLayout {
    int S;                                   // segments per sample
    int E_pad;                               // S * kSeg: row length of the decay table
    size_t dec, segm, carry, mask, counters, listed, work, pool, total;
    size_t n_counters;                       // uint32 counters reset by every call
    size_t pool_cap;                         // pool entries per sample
};
FwdLayout fwd_layout(int B, int E_max, int N, int pool_cap);

int check_params(const lif_params* p);
Model make_model(const lif_params& p);
int validate_forward_args(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                          const float* WT, int C_in, int N, const lif_params* p, const float* out_t,
                          const int32_t* out_n, const int32_t* status);
int check_launch();

// The sequential baseline (one thread per (sample, neuron), every event in
// order) on per-neuron queues (lif_forward.hip).
int launch_sequential_queue(const float* q_t, const int32_t* q_k, const int32_t* ev_src, const int32_t* ev_n, int B,
                            int E_max, const float* WT, int C_in, int N, const Model& m, float* out_t, int32_t* out_n,
                            float* out_i, int32_t* out_k, int32_t* status, hipStream_t stream);

// The chunked walk of lif_layer_forward_chunked (lif_chunked.hip), on the
// sample queues (q_k null) or on per-neuron queues (ev_t = arrival times
// [B][N][E_max], q_k = the sample's event index of each entry).
int launch_chunked_walk(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, const int32_t* q_k, int B,
                        int E_max, const float* WT, int C_in, int N, const Model& m, int K, int C, float* out_t,
                        int32_t* out_n, float* out_i, int32_t* out_k, int32_t* consumed, int32_t* processed,
                        int32_t* status, hipStream_t stream);

// The regularisers' batch terms (lif_forward.hip), shared by the plain and
// the delayed layer: from the per-(sample, neuron) hinge means ub, ob the
// two loss terms (loss nullable) and the per-neuron gates; from the interval
// counts and the gates the per-(sample, neuron) multipliers coef = (G_u, G_o)
// of the active intervals and their bound musum = |G_u| nsil + |G_o| nspk.
void launch_reg_loss(const double* ub, const double* ob, const int32_t* out_n, int B, int N, int s_max,
                     double c_target, float* loss, double2* gates, hipStream_t stream);
void launch_regg_coef(const double2* counts, const double2* gates, const int32_t* out_n, int B, int N, int s_max,
                      double c_target, double lam_reg, double lam_over, double2* coef, double* musum,
                      hipStream_t stream);

// Kernel timer (lif_timer_*): a HIP event pair per launch, recorded by the
// dispatch of the kernel itself (hipExtLaunchKernelGGL), so that the elapsed
// time is the kernel's own execution.
bool timer_events(const char* name, hipEvent_t* start, hipEvent_t* stop);
bool timer_on();

}  // namespace lif

#define TIMED_LAUNCH(name, kern, grid, block, shmem, stream, ...)                      \
    do {                                                                               \
        hipEvent_t _a, _b;                                                             \
        if (::lif::timer_on() && ::lif::timer_events(name, &_a, &_b))                  \
            hipExtLaunchKernelGGL(kern, grid, block, shmem, stream, _a, _b, 0, __VA_ARGS__); \
        else                                                                           \
            hipLaunchKernelGGL(kern, grid, block, shmem, stream, __VA_ARGS__);         \
    } while (0)
