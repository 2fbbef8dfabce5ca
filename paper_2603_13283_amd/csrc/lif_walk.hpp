// lif_walk.hpp -- segment-walk helpers shared by the forward walks
// (k_aggregate, k_check) and the backward adjoint walk (k_event_adjoint):
// work-item coordinates, per-wave staging of a segment's sources and decays,
// and the weight gather of groups of events.
#pragma once

#include "lif_common.hpp"

namespace lif {

// Workgroup index -> work index such that each of the 8 XCDs (which receive
// workgroups round-robin) processes a contiguous, sample-major range: the
// events and decays of a sample then stay in one XCD's L2.
__device__ __forceinline__ int xcd_remap(int wg, int total)
{
    int xcd = wg & 7, local = wg >> 3;
    int per = (total + 7) >> 3;
    int full = (total & 7) ? (total & 7) : 8;
    int base = xcd < full ? xcd * per : full * per + (xcd - full) * (per - 1);
    return base + local;
}

// ---------------------------------------------------------------------------
// Segment walks (k_aggregate, k_check).  A work item is (sample, segment,
// tile of 64 NPL neurons) and takes one wave; a workgroup runs kWalkWaves
// consecutive items.  Lane l holds neurons tile * 64 NPL + l NPL + i,
// i < NPL, and reads their weights of an event with one NPL-wide load from
// the event's W^T row (the wave reads 256 NPL contiguous bytes).  Sources
// and decays are wave-uniform and are read with scalar loads; the weights of
// the next kSub events are loaded while the current kSub events are walked.
// ---------------------------------------------------------------------------
constexpr int kWalkWaves = 4;

struct WalkCoords {
    int b, seg, tile, lane, n0, nb, k0, cnt;
    bool live;                    // the lane holds neurons (n0 < N)
};

template <int NPL>
__device__ __forceinline__ bool walk_coords(int items, int tiles, int S, const int32_t* __restrict__ ev_n, int E_max,
                                            int N, WalkCoords& c)
{
    // wave-uniform by construction; readfirstlane lets the compiler keep
    // everything derived from it (sources, decays) in scalar registers
    const int item = __builtin_amdgcn_readfirstlane(xcd_remap(blockIdx.x, gridDim.x) * kWalkWaves +
                                                    (int)threadIdx.x / kWave);
    if (item >= items) return false;
    c.tile = item % tiles;
    const int rest = item / tiles;
    c.seg = rest % S;
    c.b = rest / S;
    c.lane = (int)threadIdx.x % kWave;
    c.nb = clamp_count(ev_n[c.b], E_max);
    c.k0 = c.seg * kSeg;
    if (c.k0 >= c.nb) return false;
    c.cnt = min(kSeg, c.nb - c.k0);
    const int n0 = c.tile * (kWave * NPL) + c.lane * NPL;
    c.live = n0 < N;
    c.n0 = c.live ? n0 : 0;
    return true;
}

template <int NPL>
__device__ __forceinline__ void load_w(const float* __restrict__ p, float (&w)[NPL])
{
    if constexpr (NPL == 4) {
        const float4 v = *reinterpret_cast<const float4*>(p);
        w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
    } else if constexpr (NPL == 2) {
        const float2 v = *reinterpret_cast<const float2*>(p);
        w[0] = v.x; w[1] = v.y;
    } else {
        w[0] = *p;
    }
}

// Per-wave staging of a segment.  The sources of its events go to VGPRs
// (lane l holds those of events l and l + 64) and are broadcast with one lane
// read per event; the decays (A, D) and screen slopes lk go to the wave's
// slice of LDS and are read back as wave-wide broadcasts; for the check pass
// also the largest slope of each group of kGrp intervals.  The weights are
// read with buffer loads whose per-event row offset is a scalar operand, so
// a load in flight holds no address registers.
constexpr int kGrp = 8;
constexpr int kGrpPerSeg = kSeg / kGrp;
static_assert(kSub == 2 * kGrp && kWave % kGrp == 0, "a sub-block is two groups; groups tile lane ranges");
constexpr int kSrcRegs = kSeg / kWave;

struct Stage {
    int off[kSrcRegs];                 // W^T row byte offsets of events lane, lane + 64
    __amdgpu_buffer_rsrc_t rsrc;       // W^T as a raw buffer
    uint32_t lane_off;                 // byte offset of the lane's first neuron in a row
};

__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The buffer descriptor's fourth word for raw 32-bit-element buffers on gfx9.
constexpr int kRsrcWord3 = 0x00020000;

__device__ __forceinline__ Stage stage_segment(const WalkCoords& c, const int32_t* __restrict__ ss,
                                               const Decay* __restrict__ sd, const float* __restrict__ WT, int C_in,
                                               int N, double2* __restrict__ lad, double* __restrict__ llk,
                                               double* __restrict__ lgk)
{
    Stage st;
    st.rsrc = __builtin_amdgcn_make_buffer_rsrc((void*)WT, (short)0, (int)((uint32_t)C_in * (uint32_t)N * 4u),
                                                kRsrcWord3);
    st.lane_off = (uint32_t)c.n0 * 4u;
#pragma unroll
    for (int h = 0; h < kSrcRegs; ++h) {
        const int e = h * kWave + c.lane;
        st.off[h] = clamp_src(ss[min(e, c.cnt - 1)], C_in) * N * 4;
        if (sd) {                       // else the caller has filled lad
            const Decay d = sd[e];
            lad[e] = make_double2(d.A, d.D);
            if (llk) llk[e] = d.lk;
        }
    }
    wave_lds_sync();
    if (lgk) {
        if (c.lane < kGrpPerSeg) {
            double g = 0.0;
#pragma unroll
            for (int j = 0; j < kGrp; ++j) g = fmax(g, llk[c.lane * kGrp + j]);
            lgk[c.lane] = g;
        }
        wave_lds_sync();
    }
    return st;
}

template <int NPL>
__device__ __forceinline__ void load_w(const Stage& st, int soff, float (&w)[NPL])
{
    if constexpr (NPL == 4) {
        const float4 v = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(st.rsrc, st.lane_off, soff, 0));
        w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
    } else if constexpr (NPL == 2) {
        const float2 v = __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(st.rsrc, st.lane_off, soff, 0));
        w[0] = v.x; w[1] = v.y;
    } else {
        w[0] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(st.rsrc, st.lane_off, soff, 0));
    }
}

// Weights of events e0 .. e0 + kGrp - 1 of the segment (past the last event
// the last event's row is read again; the walks never use those).
template <int NPL>
__device__ __forceinline__ void load_grp(const Stage& st, int e0, float (&w)[kGrp][NPL])
{
    const int oreg = e0 < kWave ? st.off[0] : st.off[kSrcRegs - 1];
#pragma unroll
    for (int j = 0; j < kGrp; ++j) load_w<NPL>(st, __builtin_amdgcn_readlane(oreg, (e0 + j) & (kWave - 1)), w[j]);
}

// Sums over the 64 lanes of v[0..7] (one value per event of a group):
// lane l ends with the sum of v[j] for j = 4 b5 + 2 b4 + b3 (b5, b4, b3 the
// bits 5, 4, 3 of l), by a halving exchange (4 + 2 + 1 shuffles) and a
// butterfly over the lane's 8-lane row (3 shuffles).
__device__ __forceinline__ double group_sum8(const double (&v)[kGrp], int lane)
{
    const bool u32 = (lane & 32) != 0, u16 = (lane & 16) != 0, u8 = (lane & 8) != 0;
    double r4[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const double keep = u32 ? v[q + 4] : v[q], send = u32 ? v[q] : v[q + 4];
        r4[q] = keep + __shfl_xor(send, 32, kWave);
    }
    double r2[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const double keep = u16 ? r4[q + 2] : r4[q], send = u16 ? r4[q] : r4[q + 2];
        r2[q] = keep + __shfl_xor(send, 16, kWave);
    }
    double r = (u8 ? r2[1] : r2[0]) + __shfl_xor(u8 ? r2[0] : r2[1], 8, kWave);
    r += __shfl_xor(r, 4, kWave);
    r += __shfl_xor(r, 2, kWave);
    r += __shfl_xor(r, 1, kWave);
    return r;
}

}  // namespace lif
