// lif_host.hpp -- host-side helpers shared by the library's entry points:
// argument validation, model constants, workspace layout, launch timing.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#include "../../include/lif.h"
#include "lif_common.hpp"

namespace lif {

struct FwdLayout {
    int S;                                   // segments per sample
    size_t dec, segm, agg, carry, mask, winfo, counters, listed, work, pool, pool_ub, total;
    size_t pool_cap;                         // records in the pool
};
FwdLayout fwd_layout(int B, int E_max, int N);

int check_params(const lif_params* p);
Model make_model(const lif_params& p);
int validate_forward_args(const float* ev_t, const int32_t* ev_src, const int32_t* ev_n, int B, int E_max,
                          const float* WT, int C_in, int N, const lif_params* p, const float* out_t,
                          const int32_t* out_n, const int32_t* status, const void* ws);
int check_launch();

// Kernel timer (lif_timer_*): records a HIP event pair around each launch.
void timer_begin(const char* name, hipStream_t s);
void timer_end(hipStream_t s);
bool timer_on();

}  // namespace lif

#define TIMED_LAUNCH(name, kern, grid, block, shmem, stream, ...)                \
    do {                                                                         \
        bool _t = ::lif::timer_on();                                             \
        if (_t) ::lif::timer_begin(name, stream);                                \
        hipLaunchKernelGGL(kern, grid, block, shmem, stream, __VA_ARGS__);       \
        if (_t) ::lif::timer_end(stream);                                        \
    } while (0)
