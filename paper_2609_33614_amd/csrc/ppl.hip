// Perplexity signal for the threshold's performance-based adjustment
// (Sec. 3.3), gfx950.
//
// The LM-head projection z = h W_V^T runs on the dense bf16 stream / wide
// kernels (expert.hip, wide.hip) into fp32 rows (slices of the reduction
// dimension at decode sizes, added in order here).  ppl_chunk_kernel folds
// each of up to 16 vocabulary chunks of a row into an online logsumexp
// pair (running max, sum of exp(z - max)) in one pass; ppl_finish_kernel
// merges a row's chunks in order and forms NLL = logsumexp - z[target] and
// the sequence's running state in fp64: sum of NLL, token count, perplexity
// exp(sum / count) and the trend (+1 rose since the previous token, -1 did
// not, 0 first token).  Every merge has a fixed order, so results are
// bit-reproducible.
#include <math.h>

#include <algorithm>

#include "eat_device.h"
#include "eat_internal.h"

namespace eat {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kPplChunks = 16;            // vocabulary chunks per row in the logsumexp pass

// online logsumexp pair (m, s): the running max and sum of exp(z - m)
struct Lse {
    float m, s;
};

__device__ __forceinline__ Lse lse_merge(Lse a, Lse b) {
    if (a.m < b.m) { const Lse t = a; a = b; b = t; }
    if (b.m == -INFINITY) return a;
    return {a.m, a.s + b.s * expf(b.m - a.m)};
}

// logit j of a row: the GEMM's reduction slices added in slice order
__device__ __forceinline__ float logit(const float* row, int splits, int64_t stride, int j) {
    float v = row[j];
    for (int sp = 1; sp < splits; ++sp) v += row[sp * stride + j];
    return v;
}

// grid (S, chunks): each workgroup folds one chunk of a row into an (m, s)
// pair in one pass; lanes by stride, then the wave by butterfly, then the
// waves in order.
__global__ __launch_bounds__(kThreads) void ppl_chunk_kernel(const float* __restrict__ z, int splits, int64_t stride,
                                                             int V, int chunk, float2* __restrict__ part) {
    __shared__ Lse red[kWaves];
    const int s = blockIdx.x, c = blockIdx.y;
    const float* row = z + static_cast<size_t>(s) * V;
    const int j0 = c * chunk, j1 = min(V, j0 + chunk);
    Lse a{-INFINITY, 0.f};
    for (int j = j0 + threadIdx.x; j < j1; j += kThreads) {
        const float v = logit(row, splits, stride, j);
        if (v > a.m) { a.s = a.s * expf(a.m - v) + 1.f; a.m = v; }
        else a.s += expf(v - a.m);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const Lse b{__shfl_xor(a.m, off, kWave), __shfl_xor(a.s, off, kWave)};
        // merge in a fixed (lower lane first) order so partners agree bit for bit
        a = (lane_id() & off) ? lse_merge(b, a) : lse_merge(a, b);
    }
    if (lane_id() == 0) red[threadIdx.x / kWave] = a;
    __syncthreads();
    if (threadIdx.x != 0) return;
    Lse t = red[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) t = lse_merge(t, red[w]);
    part[static_cast<size_t>(s) * gridDim.y + c] = make_float2(t.m, t.s);
}

// one thread per sequence: chunks merged in order, NLL, running state, trend
__global__ __launch_bounds__(kThreads) void ppl_finish_kernel(const float* __restrict__ z, int splits,
                                                              int64_t stride, int S, int V, int chunks,
                                                              const float2* __restrict__ part,
                                                              const int32_t* __restrict__ target, double* nll_sum,
                                                              int32_t* count, double* ppl_prev, int8_t* trend,
                                                              float* nll_out) {
    const int s = blockIdx.x * kThreads + threadIdx.x;
    if (s >= S) return;
    Lse t{-INFINITY, 0.f};
    for (int c = 0; c < chunks; ++c) {
        const float2 q = part[static_cast<size_t>(s) * chunks + c];
        t = lse_merge(t, Lse{q.x, q.y});
    }
    const int y = target[s];
    double nll = NAN;
    if (y >= 0 && y < V)
        nll = static_cast<double>(t.m) + log(static_cast<double>(t.s)) -
              static_cast<double>(logit(z + static_cast<size_t>(s) * V, splits, stride, y));
    const double sum = nll_sum[s] + nll;
    const int32_t n = count[s] + 1;
    const double ppl = exp(sum / n);
    trend[s] = n > 1 ? (ppl > ppl_prev[s] ? 1 : -1) : 0;
    nll_sum[s] = sum;
    count[s] = n;
    ppl_prev[s] = ppl;
    if (nll_out) nll_out[s] = static_cast<float>(nll);
}

__global__ __launch_bounds__(kThreads) void ppl_reset_kernel(int S, double* nll_sum, int32_t* count,
                                                             double* ppl_prev) {
    const int s = blockIdx.x * kThreads + threadIdx.x;
    if (s < S) { nll_sum[s] = 0.0; count[s] = 0; ppl_prev[s] = 0.0; }
}

}  // namespace

int ppl_chunks(int V) { return std::min(kPplChunks, (V + kThreads - 1) / kThreads); }

hipError_t launch_ppl(const float* z, int splits, int64_t stride, int32_t S, int V, const int32_t* target,
                      double* nll_sum, int32_t* count, double* ppl_prev, int8_t* trend, float* nll_out,
                      float2* part, hipStream_t s) {
    const int chunks = ppl_chunks(V);
    const int chunk = (V + chunks - 1) / chunks;
    ppl_chunk_kernel<<<dim3(S, chunks), kThreads, 0, s>>>(z, splits, stride, V, chunk, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    ppl_finish_kernel<<<(S + kThreads - 1) / kThreads, kThreads, 0, s>>>(z, splits, stride, S, V, chunks, part, target,
                                                                         nll_sum, count, ppl_prev, trend, nll_out);
    return hipGetLastError();
}

// Reduction slices of the LM-head GEMM: the dense heuristic, capped (each
// slice costs one more S x V fp32 read in the logsumexp).
#ifndef EAT_PPL_SPLITS_MAX
#define EAT_PPL_SPLITS_MAX 2
#endif
int ppl_splits(int32_t S, int d, int V) { return std::min(dense_splits(V, d, S), EAT_PPL_SPLITS_MAX); }

hipError_t launch_ppl_reset(int32_t S, double* nll_sum, int32_t* count, double* ppl_prev, hipStream_t s) {
    ppl_reset_kernel<<<(S + kThreads - 1) / kThreads, kThreads, 0, s>>>(S, nll_sum, count, ppl_prev);
    return hipGetLastError();
}

}  // namespace eat
