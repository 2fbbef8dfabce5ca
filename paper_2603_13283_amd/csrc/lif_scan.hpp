// lif_scan.hpp -- wave-wide scans of affine maps x -> a x + b (the event
// maps of App. B form a semigroup under composition) with DPP row shifts
// inside each row of 16 lanes and lane reads across the four rows, instead
// of LDS-crossbar lane permutes.
#pragma once

#include "lif_common.hpp"

namespace lif {

// v of lane j -/+ Dist within the calling lane's row of 16 lanes (DPP row
// shift right / left); lanes without a source get fill.
template <int Ctrl>
__device__ __forceinline__ double dpp_double(double v, double fill)
{
    const unsigned long long u = (unsigned long long)__double_as_longlong(v);
    const unsigned long long f = (unsigned long long)__double_as_longlong(fill);
    const unsigned lo = (unsigned)__builtin_amdgcn_update_dpp((int)(unsigned)f, (int)(unsigned)u, Ctrl, 0xf, 0xf,
                                                              false);
    const unsigned hi = (unsigned)__builtin_amdgcn_update_dpp((int)(unsigned)(f >> 32), (int)(unsigned)(u >> 32),
                                                              Ctrl, 0xf, 0xf, false);
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// v of lane j - 1 (lane 0: fill) / of lane j + 1 (lane 63: fill) across the
// whole wave (DPP wave shifts).
__device__ __forceinline__ double wave_shr1(double v, double fill) { return dpp_double<0x138>(v, fill); }
__device__ __forceinline__ double wave_shl1(double v, double fill) { return dpp_double<0x130>(v, fill); }

// v of lane l (l wave-uniform).
__device__ __forceinline__ double read_lane_double(double v, int l)
{
    const unsigned long long u = (unsigned long long)__double_as_longlong(v);
    const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)u, l);
    const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(u >> 32), l);
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// Inclusive scan upwards: lane j ends with the composition of the maps of
// lanes 0 .. j (lane j's applied last).
__device__ __forceinline__ void scan_maps_up(double& a, double& b, int lane)
{
    auto step = [&](double pa, double pb) {
        b = fma(a, pb, b);
        a *= pa;
    };
    step(dpp_double<0x111>(a, 1.0), dpp_double<0x111>(b, 0.0));
    step(dpp_double<0x112>(a, 1.0), dpp_double<0x112>(b, 0.0));
    step(dpp_double<0x114>(a, 1.0), dpp_double<0x114>(b, 0.0));
    step(dpp_double<0x118>(a, 1.0), dpp_double<0x118>(b, 0.0));
    const int row = lane >> 4;
    {   // rows 1 and 3 after the totals of rows 0 and 2
        const double a15 = read_lane_double(a, 15), b15 = read_lane_double(b, 15);
        const double a47 = read_lane_double(a, 47), b47 = read_lane_double(b, 47);
        if (row & 1) step(row == 1 ? a15 : a47, row == 1 ? b15 : b47);
    }
    {   // rows 2 and 3 after the total of lanes 0 .. 31
        const double a31 = read_lane_double(a, 31), b31 = read_lane_double(b, 31);
        if (row >= 2) step(a31, b31);
    }
}

// Inclusive scan downwards: lane j ends with the composition of the maps of
// lanes j .. 63 (lane j's applied last).
__device__ __forceinline__ void scan_maps_down(double& a, double& b, int lane)
{
    auto step = [&](double pa, double pb) {
        b = fma(a, pb, b);
        a *= pa;
    };
    step(dpp_double<0x101>(a, 1.0), dpp_double<0x101>(b, 0.0));
    step(dpp_double<0x102>(a, 1.0), dpp_double<0x102>(b, 0.0));
    step(dpp_double<0x104>(a, 1.0), dpp_double<0x104>(b, 0.0));
    step(dpp_double<0x108>(a, 1.0), dpp_double<0x108>(b, 0.0));
    const int row = lane >> 4;
    {   // rows 0 and 2 before the totals of rows 1 and 3
        const double a16 = read_lane_double(a, 16), b16 = read_lane_double(b, 16);
        const double a48 = read_lane_double(a, 48), b48 = read_lane_double(b, 48);
        if (!(row & 1)) step(row == 0 ? a16 : a48, row == 0 ? b16 : b48);
    }
    {   // rows 0 and 1 before the total of lanes 32 .. 63
        const double a32 = read_lane_double(a, 32), b32 = read_lane_double(b, 32);
        if (row < 2) step(a32, b32);
    }
}

}  // namespace lif
