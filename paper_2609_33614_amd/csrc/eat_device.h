// Device-side helpers shared by the gfx950 kernels of the EAT layer.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace eat {

constexpr int kWave = 64;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Reductions over the 64 lanes of a wave.  Inside each 16-lane row, DPP
// lane swaps (neighbour pairs, quad pairs, then the 8-lane and 16-lane
// mirrors) leave every lane of the row holding the row's total -- the
// partners add a commutative pair, so the row's lanes agree bit for bit;
// then the four row totals, read through SGPRs, are combined in a fixed
// order.  Every lane ends with the same value, the order of operations never
// depends on timing, and no step goes through LDS (a ds_bpermute butterfly
// costs an LDS round trip per step).
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
    return __builtin_amdgcn_update_dpp(v, v, CTRL, 0xf, 0xf, false);
}
constexpr int kDppXor1 = 0xB1;          // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;          // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;   // lane i <-> 7 - i within 8
constexpr int kDppMirror = 0x140;       // lane i <-> 15 - i within 16

template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
    return __int_as_float(dpp_i<CTRL>(__float_as_int(v)));
}
template <int CTRL>
__device__ __forceinline__ double dpp_d(double v) {
    const int lo = dpp_i<CTRL>(__double2loint(v)), hi = dpp_i<CTRL>(__double2hiint(v));
    return __hiloint2double(hi, lo);
}
__device__ __forceinline__ float lane_f(float v, int j) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), j));
}
__device__ __forceinline__ double lane_d(double v, int j) {
    return __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(v), j),
                            __builtin_amdgcn_readlane(__double2loint(v), j));
}

__device__ __forceinline__ float wave_sum(float v) {
    v += dpp_f<kDppXor1>(v);
    v += dpp_f<kDppXor2>(v);
    v += dpp_f<kDppHalfMirror>(v);
    v += dpp_f<kDppMirror>(v);
    return (lane_f(v, 0) + lane_f(v, 16)) + (lane_f(v, 32) + lane_f(v, 48));
}
__device__ __forceinline__ double wave_sum(double v) {
    v += dpp_d<kDppXor1>(v);
    v += dpp_d<kDppXor2>(v);
    v += dpp_d<kDppHalfMirror>(v);
    v += dpp_d<kDppMirror>(v);
    return (lane_d(v, 0) + lane_d(v, 16)) + (lane_d(v, 32) + lane_d(v, 48));
}
__device__ __forceinline__ int wave_sum(int v) {
    v += dpp_i<kDppXor1>(v);
    v += dpp_i<kDppXor2>(v);
    v += dpp_i<kDppHalfMirror>(v);
    v += dpp_i<kDppMirror>(v);
    return (__builtin_amdgcn_readlane(v, 0) + __builtin_amdgcn_readlane(v, 16)) +
           (__builtin_amdgcn_readlane(v, 32) + __builtin_amdgcn_readlane(v, 48));
}
__device__ __forceinline__ float wave_max(float v) {
    v = fmaxf(v, dpp_f<kDppXor1>(v));
    v = fmaxf(v, dpp_f<kDppXor2>(v));
    v = fmaxf(v, dpp_f<kDppHalfMirror>(v));
    v = fmaxf(v, dpp_f<kDppMirror>(v));
    return fmaxf(fmaxf(lane_f(v, 0), lane_f(v, 16)), fmaxf(lane_f(v, 32), lane_f(v, 48)));
}

// Tile table of expert-major row segments: tstart[g] = sum over h < g of
// ceil((offsets[h+1] - offsets[h]) / bm), for g = 0..groups.  Wave 0 reads
// one segment per lane and scans 64 at a time (integer sums, so the order
// does not matter); every thread of the workgroup must call it.  With
// COUNT, `used` (LDS) receives the number of non-empty segments.
template <bool COUNT = false>
__device__ __forceinline__ void tile_starts(const int32_t* offsets, int groups, int bm, int* tstart,
                                            int* used = nullptr) {
    if (threadIdx.x < kWave) {
        const int lane = __lane_id();
        int carry = 0, nonempty = 0;
        for (int g0 = 0; g0 < groups; g0 += kWave) {
            const int g = g0 + lane;
            int c = g < groups ? (offsets[g + 1] - offsets[g] + bm - 1) / bm : 0;
            if constexpr (COUNT) nonempty += __popcll(__ballot(c > 0));
#pragma unroll
            for (int o = 1; o < kWave; o <<= 1) {
                const int u = __shfl_up(c, o, kWave);
                if (lane >= o) c += u;
            }
            if (g < groups) tstart[g + 1] = carry + c;
            carry += __shfl(c, kWave - 1, kWave);
        }
        if (lane == 0) {
            tstart[0] = 0;
            if constexpr (COUNT) *used = nonempty;
        }
    }
    __syncthreads();
}

// Segment holding tile `tile` (0 <= tile < tstart[groups]): the first g with
// tstart[g + 1] > tile, by binary search (empty segments are skipped).
__device__ __forceinline__ int tile_group(const int* tstart, int groups, int tile) {
    int lo = 0, hi = groups - 1;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (tstart[mid + 1] > tile) hi = mid;
        else lo = mid + 1;
    }
    return lo;
}

// Broadcast lane j's value (j uniform across the wave) through an SGPR.
__device__ __forceinline__ float read_lane(float v, int j) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), j));
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}
// Round-to-nearest-even fp32 -> bf16 bits; a NaN stays a (quiet) NaN.
// Written as a select, not a branch, so that converting a tile of results
// stays straight-line code.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    const uint32_t u = __float_as_uint(f);
    const uint32_t rne = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
    const uint32_t qnan = (u >> 16) | 0x40u;
    return static_cast<uint16_t>((u & 0x7fffffffu) > 0x7f800000u ? qnan : rne);
}

// Two fp32 values -> packed bf16 bits (a in the low half), round to nearest
// even by the hardware conversion (one instruction; NaN stays NaN).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, bf16x2));
}

__device__ __forceinline__ float silu(float a) { return a / (1.0f + __expf(-a)); }

// Workgroup barrier that only waits for this wave's LDS traffic.  Global
// loads issued before it stay in flight (__syncthreads() would drain them
// with a full fence); the "memory" clobber keeps the compiler from moving
// LDS accesses across it.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Wait until at most N vector-memory operations of this wave are
// outstanding (vmcnt(N); expcnt and lgkmcnt left unconstrained, gfx9
// encoding).  Loads complete in issue order for this counter, so a count of
// the loads issued after the one awaited names it exactly.
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

}  // namespace eat
