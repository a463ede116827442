// Combine and account kernels (gfx950).
//
// combine: one workgroup per token gathers the token's expert rows in
// increasing expert order, adds the split-K partials of each row (in split
// order), writes ||o||_2 of every un-gated row, and accumulates
// y_t = sum_e g_norm,t,e o_t,e (+ shared expert) in fp32 (Eq. 7-8 and the
// weighted fusion of Sec. 3.4).  No atomics: every output element has one
// writer and a fixed summation order.
//
// accounts: one wave per expert reduces its contiguous row segment in fp64
// and applies the Sec. 3.2 bookkeeping once per call:
//   N += n_e,  P_total += sum of the rows' router probabilities,
//   C_s = (1 - alpha) C_s + alpha * mean row norm.
#include <math.h>

#include "eat_device.h"
#include "eat_internal.h"

namespace eat {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;

struct CombineArgs {
    const uint64_t* mask;
    const float* gate;
    const int32_t* inv;
    const float* yp;           // [splits][rows_cap][d]
    const float* ys;           // [T][d] shared output or null
    void* y;
    float* nrm;
    int64_t split_stride;
    int splits, T, E, d;
};

template <typename YT, int NV>
__global__ __launch_bounds__(kThreads) void combine_kernel(CombineArgs a) {
    __shared__ float red[kWaves];
    const int t = blockIdx.x;
    const int lane = lane_id(), wave = threadIdx.x / kWave;
    const int nvec = a.d / 4;
    float4 acc[NV];
#pragma unroll
    for (int v = 0; v < NV; ++v) acc[v] = make_float4(0.f, 0.f, 0.f, 0.f);

    const uint64_t m = a.mask[t];
    for (uint64_t rest = m; rest; rest &= rest - 1) {
        const int e = __builtin_ctzll(rest);
        const int64_t row = a.inv[static_cast<size_t>(t) * a.E + e];
        const float g = a.gate[static_cast<size_t>(t) * a.E + e];
        float ss = 0.f;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            const int j = threadIdx.x + v * kThreads;
            if (j >= nvec) break;
            const float* src = a.yp + row * a.d + 4 * j;
            float4 o = *reinterpret_cast<const float4*>(src);
            for (int sp = 1; sp < a.splits; ++sp) {
                const float4 q = *reinterpret_cast<const float4*>(src + sp * a.split_stride);
                o.x += q.x; o.y += q.y; o.z += q.z; o.w += q.w;
            }
            ss = fmaf(o.x, o.x, ss); ss = fmaf(o.y, o.y, ss);
            ss = fmaf(o.z, o.z, ss); ss = fmaf(o.w, o.w, ss);
            acc[v].x = fmaf(g, o.x, acc[v].x); acc[v].y = fmaf(g, o.y, acc[v].y);
            acc[v].z = fmaf(g, o.z, acc[v].z); acc[v].w = fmaf(g, o.w, acc[v].w);
        }
        ss = wave_sum(ss);
        if (lane == 0) red[wave] = ss;
        __syncthreads();
        if (threadIdx.x == 0) {
            float tot = 0.f;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) tot += red[w];
            a.nrm[row] = sqrtf(tot);
        }
        __syncthreads();
    }
#pragma unroll
    for (int v = 0; v < NV; ++v) {
        const int j = threadIdx.x + v * kThreads;
        if (j >= nvec) break;
        float4 r = acc[v];
        if (a.ys) {
            const float4 q = *reinterpret_cast<const float4*>(a.ys + static_cast<size_t>(t) * a.d + 4 * j);
            r.x += q.x; r.y += q.y; r.z += q.z; r.w += q.w;
        }
        if constexpr (sizeof(YT) == 4) {
            *reinterpret_cast<float4*>(static_cast<float*>(a.y) + static_cast<size_t>(t) * a.d + 4 * j) = r;
        } else {
            uint2 pk;
            pk.x = static_cast<uint32_t>(f32_to_bf16(r.x)) | (static_cast<uint32_t>(f32_to_bf16(r.y)) << 16);
            pk.y = static_cast<uint32_t>(f32_to_bf16(r.z)) | (static_cast<uint32_t>(f32_to_bf16(r.w)) << 16);
            *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.y) + static_cast<size_t>(t) * a.d + 4 * j) = pk;
        }
    }
}

template <typename YT>
hipError_t launch_combine_t(const CombineArgs& a, hipStream_t s) {
    const int nv = (a.d / 4 + kThreads - 1) / kThreads;
    if (nv <= 1) combine_kernel<YT, 1><<<a.T, kThreads, 0, s>>>(a);
    else if (nv <= 2) combine_kernel<YT, 2><<<a.T, kThreads, 0, s>>>(a);
    else if (nv <= 4) combine_kernel<YT, 4><<<a.T, kThreads, 0, s>>>(a);
    else combine_kernel<YT, 8><<<a.T, kThreads, 0, s>>>(a);
    return hipGetLastError();
}

__global__ __launch_bounds__(kWave) void update_accounts_kernel(
    const int32_t* __restrict__ offsets, const int32_t* __restrict__ tok_idx,
    const float* __restrict__ prob, const float* __restrict__ nrm, int E, float alpha,
    int64_t* __restrict__ n, float* __restrict__ p_total, float* __restrict__ c_s) {
    const int e = blockIdx.x;
    const int lane = lane_id();
    const int beg = offsets[e], end = offsets[e + 1];
    const int cnt = end - beg;
    if (cnt <= 0) return;
    double sp = 0.0, sn = 0.0;
    for (int r = beg + lane; r < end; r += kWave) {
        sp += static_cast<double>(prob[static_cast<size_t>(tok_idx[r]) * E + e]);
        sn += static_cast<double>(nrm[r]);
    }
    sp = wave_sum(sp);
    sn = wave_sum(sn);
    if (lane == 0) {
        n[e] += cnt;
        p_total[e] = static_cast<float>(static_cast<double>(p_total[e]) + sp);
        const double a = static_cast<double>(alpha);
        c_s[e] = static_cast<float>((1.0 - a) * static_cast<double>(c_s[e]) + a * (sn / cnt));
    }
}

__global__ __launch_bounds__(kWave) void reset_accounts_kernel(int E, int64_t* n, float* p, float* c) {
    const int e = lane_id();
    if (e < E) { n[e] = 0; p[e] = 0.f; c[e] = 0.f; }
}

}  // namespace

hipError_t launch_combine(const eat_params_t& p, int32_t T, const uint64_t* mask, const float* gate,
                          const int32_t* inv, const float* yp, const float* ys, void* y, float* nrm,
                          int splits, int64_t split_stride, hipStream_t s) {
    CombineArgs a{mask, gate, inv, yp, ys, y, nrm, split_stride, splits, T, p.E, p.d_model};
    if (p.act_dtype == EAT_BF16) return launch_combine_t<uint16_t>(a, s);
    return launch_combine_t<float>(a, s);
}

hipError_t launch_update_accounts(const eat_params_t& p, const int32_t* offsets, const int32_t* tok_idx,
                                  const float* prob, const float* nrm, eat_accounts_t acc, hipStream_t s) {
    update_accounts_kernel<<<p.E, kWave, 0, s>>>(offsets, tok_idx, prob, nrm, p.E, p.alpha, acc.n,
                                                 acc.p_total, acc.c_s);
    return hipGetLastError();
}

hipError_t launch_reset_accounts(const eat_params_t& p, eat_accounts_t acc, hipStream_t s) {
    reset_accounts_kernel<<<1, kWave, 0, s>>>(p.E, acc.n, acc.p_total, acc.c_s);
    return hipGetLastError();
}

}  // namespace eat
