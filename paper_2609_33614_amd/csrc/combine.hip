// Combine, account and stacked-layer kernels (gfx950).
//
// combine: per token and 1024-element slice of d, gathers the token's expert
// rows in increasing expert order, adds the split-K partials of each row (in
// split order), writes each row slice's sum of squares, and accumulates
// y_t = sum_e g_norm,t,e o_t,e (+ shared expert) (+ a residual row) in fp32
// (Eq. 7-8 and the weighted fusion of Sec. 3.4).  After a prefill-sized down
// projection the rows come in bf16 with their sums of squares already taken
// (from the projection's fp32 accumulators), which halves the bytes read;
// combine_rows16_kernel gathers those, 8 elements a thread.  No atomics:
// every output element has one writer and a fixed summation order.
//
// mix_norm: between stacked layers, h' = bf16(sum of the mixing GEMM's
// split partials) and the next layer's input u = bf16(h' / rms(h')), one
// workgroup per token.
//
// accounts: the Sec. 3.2 bookkeeping once per call, each expert's contiguous
// row segment reduced in fp64:
//   N += n_e,  P_total += sum of the rows' router probabilities,
//   C_s = (1 - alpha) C_s + alpha * mean row norm,
// each row norm being sqrt of its partial sums of squares (the combine's
// slices, or the prefill down projection's 32-feature parts) added in order.
// (Doing it in the combine's last workgroup to finish instead of a kernel of
// its own needs a device-wide release in every combine workgroup, an L2
// write-back on this part: measured slower at every decode size.)
#include <math.h>

#include "eat_device.h"
#include "eat_internal.h"

namespace eat {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;

struct CombineArgs {
    const uint64_t* mask;      // [T][words]
    const float* gate;
    const int32_t* inv;
    const void* yp;            // fp32 [splits][rows_cap][d], or bf16 [rows_cap][d] (combine_rows16_kernel)
    const int32_t* splits_dev; // slices the down projection took (device), or null: `splits`
    const float* ys;           // [T][d] shared output or null
    const uint16_t* res;       // [T][d] bf16 residual rows added to y, or null
    void* y;
    float* nrm2;               // [rows_cap][nchunk] partial sums of squares
    int64_t split_stride;
    int splits, T, E, d, nchunk, words;
};

// One workgroup per (token, 1024-element slice of d): 4 elements per
// thread.  The token's experts are taken in increasing index order, up to
// kBatch at a time: every row slice of a batch is loaded (its split partials
// added in slice order) before any reduction, then the batch's sums of
// squares are reduced together (per wave by butterfly, over the waves in
// order, one barrier pair per batch) into nrm2[row][slice] (added up, in
// slice order, by the account kernel).
constexpr int kBatch = 8;
constexpr int kMaxSplits = 8;                  // the down projection uses at most 8 slices

template <typename YT>
__global__ __launch_bounds__(kThreads) void combine_kernel(CombineArgs a) {
    __shared__ float red[kBatch][kWaves];
    const int t = blockIdx.x, chunk = blockIdx.y;
    // an unconditional load (from a stand-in address when the count is the
    // host's), issued with the mask load below and waited for once
    const int sdev = *(a.splits_dev ? a.splits_dev : reinterpret_cast<const int32_t*>(a.mask));
    const int splits = a.splits_dev ? sdev : a.splits;
    const int lane = lane_id(), wave = threadIdx.x / kWave;
    const int j = chunk * kThreads + threadIdx.x;      // float4 index within the row
    const bool on = 4 * j < a.d;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    const uint64_t* mt = a.mask + static_cast<size_t>(t) * a.words;
    // the shared-expert and residual slices do not depend on the routing, so
    // they are loaded first, from in-bounds stand-ins when absent (row 0 of
    // the partials, at least d floats; element 0 for threads past d), and
    // used after the loop
    const int jc = on ? j : 0;
    const float* ypf = static_cast<const float*>(a.yp);
    const float4 ysv =
        *reinterpret_cast<const float4*>((a.ys ? a.ys + static_cast<size_t>(t) * a.d : ypf) + 4 * jc);
    const uint2 rsv = *reinterpret_cast<const uint2*>(
        (a.res ? a.res + static_cast<size_t>(t) * a.d : reinterpret_cast<const uint16_t*>(ypf)) + 4 * jc);

    int w = 0;
    uint64_t rest = mt[0];
    for (;;) {
        // next batch of selected experts (uniform across the workgroup)
        int rows[kBatch];                     // < 2^31: the row count is checked at creation
        float gs[kBatch];
        int nb = 0;
#pragma unroll
        for (int b = 0; b < kBatch; ++b) {
            while (rest == 0 && w + 1 < a.words) rest = mt[++w];
            rows[b] = 0;
            gs[b] = 0.f;
            if (rest != 0) {
                const int e = 64 * w + __builtin_ctzll(rest);
                rest &= rest - 1;
                rows[b] = a.inv[static_cast<size_t>(t) * a.E + e];
                gs[b] = a.gate[static_cast<size_t>(t) * a.E + e];
                nb = b + 1;
            }
        }
        if (nb == 0) break;
        // each row slice's partials are all loaded at once and added in slice
        // order; the next row's loads are issued before this row is added up
        // (threads past d read the row's first elements and discard them)
        constexpr int kS = kMaxSplits;
        float4 q[2][kS];
        auto issue = [&](float4 (&dst)[kS], int row) __attribute__((always_inline)) {
            const float* src = ypf + static_cast<int64_t>(row) * a.d + 4 * jc;
#pragma unroll
            for (int sp = 0; sp < kMaxSplits; ++sp)
                if (sp < splits) dst[sp] = *reinterpret_cast<const float4*>(src + sp * a.split_stride);
        };
        issue(q[0], rows[0]);
        float ss[kBatch];
#pragma unroll
        for (int b = 0; b < kBatch; ++b) {
            ss[b] = 0.f;
            if (b < nb) {
                if (b + 1 < nb) issue(q[(b + 1) & 1], rows[b + 1]);
                const float4 (&c)[kS] = q[b & 1];
                float4 o = c[0];
#pragma unroll
                for (int sp = 1; sp < kS; ++sp)
                    if (sp < splits) { o.x += c[sp].x; o.y += c[sp].y; o.z += c[sp].z; o.w += c[sp].w; }
                if (on) {
                    ss[b] = fmaf(o.x, o.x, ss[b]); ss[b] = fmaf(o.y, o.y, ss[b]);
                    ss[b] = fmaf(o.z, o.z, ss[b]); ss[b] = fmaf(o.w, o.w, ss[b]);
                    const float g = gs[b];
                    acc.x = fmaf(g, o.x, acc.x); acc.y = fmaf(g, o.y, acc.y);
                    acc.z = fmaf(g, o.z, acc.z); acc.w = fmaf(g, o.w, acc.w);
                }
            }
        }
#pragma unroll
        for (int b = 0; b < kBatch; ++b) {
            if (b >= nb) break;
            const float v = wave_sum(ss[b]);
            if (lane == 0) red[b][wave] = v;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
#pragma unroll
            for (int b = 0; b < kBatch; ++b) {
                if (b >= nb) break;
                float tot = 0.f;
#pragma unroll
                for (int q = 0; q < kWaves; ++q) tot += red[b][q];
                a.nrm2[static_cast<int64_t>(rows[b]) * a.nchunk + chunk] = tot;
            }
        }
        __syncthreads();
        if (nb < kBatch) break;
    }
    if (on) {
        if (a.ys) {
            const float4 q = ysv;
            acc.x += q.x; acc.y += q.y; acc.z += q.z; acc.w += q.w;
        }
        if (a.res) {
            const uint2 q = rsv;
            acc.x += bf16_to_f32(static_cast<uint16_t>(q.x & 0xffffu));
            acc.y += bf16_to_f32(static_cast<uint16_t>(q.x >> 16));
            acc.z += bf16_to_f32(static_cast<uint16_t>(q.y & 0xffffu));
            acc.w += bf16_to_f32(static_cast<uint16_t>(q.y >> 16));
        }
        if constexpr (sizeof(YT) == 4) {
            *reinterpret_cast<float4*>(static_cast<float*>(a.y) + static_cast<size_t>(t) * a.d + 4 * j) = acc;
        } else {
            uint2 pk;
            pk.x = static_cast<uint32_t>(f32_to_bf16(acc.x)) | (static_cast<uint32_t>(f32_to_bf16(acc.y)) << 16);
            pk.y = static_cast<uint32_t>(f32_to_bf16(acc.z)) | (static_cast<uint32_t>(f32_to_bf16(acc.w)) << 16);
            *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.y) + static_cast<size_t>(t) * a.d + 4 * j) = pk;
        }
    }
}

// After a prefill-sized down projection: the expert rows come in bf16, one
// slice, their sums of squares already taken (from the projection's fp32
// accumulators), so this pass only gathers and weights them: one workgroup
// per (token, 2048-element slice of d), 8 elements a thread (16-byte loads),
// every row of a batch of the token's experts loaded before the first is
// added; the same order of additions as combine_kernel.  y is bf16.
constexpr int kRowVec = 8;
__global__ __launch_bounds__(kThreads) void combine_rows16_kernel(CombineArgs a) {
    const int t = blockIdx.x;
    const int j = blockIdx.y * kThreads + threadIdx.x;     // 8-element group of the row
    const bool on = kRowVec * j < a.d;
    const int jc = on ? j : 0;
    const uint16_t* yph = static_cast<const uint16_t*>(a.yp);
    const uint64_t* mt = a.mask + static_cast<size_t>(t) * a.words;
    // shared-expert and residual slices first, from in-bounds stand-ins when
    // absent (expert row 0: the rows hold at least 2 d elements on this path)
    const float* ysr = a.ys ? a.ys + static_cast<size_t>(t) * a.d : reinterpret_cast<const float*>(yph);
    const float4 ys0 = *reinterpret_cast<const float4*>(ysr + kRowVec * jc);
    const float4 ys1 = *reinterpret_cast<const float4*>(ysr + kRowVec * jc + 4);
    const uint4 rsv = *reinterpret_cast<const uint4*>((a.res ? a.res + static_cast<size_t>(t) * a.d : yph) +
                                                      kRowVec * jc);
    float acc[kRowVec];
#pragma unroll
    for (int i = 0; i < kRowVec; ++i) acc[i] = 0.f;
    auto unpack = [](const uint4& q, float (&v)[kRowVec]) __attribute__((always_inline)) {
        const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[2 * i] = bf16_to_f32(static_cast<uint16_t>(w[i] & 0xffffu));
            v[2 * i + 1] = bf16_to_f32(static_cast<uint16_t>(w[i] >> 16));
        }
    };
    int w = 0;
    uint64_t rest = mt[0];
    for (;;) {
        int rows[kBatch];
        float gs[kBatch];
        int nb = 0;
#pragma unroll
        for (int b = 0; b < kBatch; ++b) {
            while (rest == 0 && w + 1 < a.words) rest = mt[++w];
            rows[b] = 0;
            gs[b] = 0.f;
            if (rest != 0) {
                const int e = 64 * w + __builtin_ctzll(rest);
                rest &= rest - 1;
                rows[b] = a.inv[static_cast<size_t>(t) * a.E + e];
                gs[b] = a.gate[static_cast<size_t>(t) * a.E + e];
                nb = b + 1;
            }
        }
        if (nb == 0) break;
        // (rows past nb read row 0, unused)
        uint4 q[kBatch];
#pragma unroll
        for (int b = 0; b < kBatch; ++b)
            q[b] = *reinterpret_cast<const uint4*>(yph + static_cast<int64_t>(rows[b]) * a.d + kRowVec * jc);
#pragma unroll
        for (int b = 0; b < kBatch; ++b) {
            if (b >= nb) break;
            float v[kRowVec];
            unpack(q[b], v);
            const float g = gs[b];
#pragma unroll
            for (int i = 0; i < kRowVec; ++i) acc[i] = fmaf(g, v[i], acc[i]);
        }
        if (nb < kBatch) break;
    }
    if (!on) return;
    if (a.ys) {
        acc[0] += ys0.x; acc[1] += ys0.y; acc[2] += ys0.z; acc[3] += ys0.w;
        acc[4] += ys1.x; acc[5] += ys1.y; acc[6] += ys1.z; acc[7] += ys1.w;
    }
    if (a.res) {
        float r[kRowVec];
        unpack(rsv, r);
#pragma unroll
        for (int i = 0; i < kRowVec; ++i) acc[i] += r[i];
    }
    uint4 pk;
    pk.x = static_cast<uint32_t>(f32_to_bf16(acc[0])) | (static_cast<uint32_t>(f32_to_bf16(acc[1])) << 16);
    pk.y = static_cast<uint32_t>(f32_to_bf16(acc[2])) | (static_cast<uint32_t>(f32_to_bf16(acc[3])) << 16);
    pk.z = static_cast<uint32_t>(f32_to_bf16(acc[4])) | (static_cast<uint32_t>(f32_to_bf16(acc[5])) << 16);
    pk.w = static_cast<uint32_t>(f32_to_bf16(acc[6])) | (static_cast<uint32_t>(f32_to_bf16(acc[7])) << 16);
    *reinterpret_cast<uint4*>(static_cast<uint16_t*>(a.y) + static_cast<size_t>(t) * a.d + kRowVec * j) = pk;
}

// Expert e's account update by one workgroup (every thread of it calls this).
__device__ __forceinline__ void account_update(const AccountJob& j, int e) {
    __shared__ double red[2][kWaves];
    const int32_t* __restrict__ offsets = j.offsets;
    const int32_t* __restrict__ tok_idx = j.tok_idx;
    const float* __restrict__ prob = j.prob;
    const float* __restrict__ nrm2 = j.nrm2;
    const int nchunk = j.parts, E = j.experts;
    const float alpha = j.alpha;
    int64_t* __restrict__ n = j.acc.n;
    float* __restrict__ p_total = j.acc.p_total;
    float* __restrict__ c_s = j.acc.c_s;
    const int lane = lane_id(), wave = threadIdx.x / kWave;
    const int beg = offsets[e], end = offsets[e + 1];
    const int cnt = end - beg;
    if (cnt <= 0) return;
    double sp = 0.0, sn = 0.0;
    for (int r = beg + threadIdx.x; r < end; r += kThreads) {
        sp += static_cast<double>(prob[static_cast<size_t>(tok_idx[r]) * E + e]);
        float ss = 0.f;
        const float* rp = nrm2 + static_cast<size_t>(r) * nchunk;
        if ((nchunk & 3) == 0) {
            // (the same order, four partials per load)
            for (int c = 0; c < nchunk; c += 4) {
                const float4 v = *reinterpret_cast<const float4*>(rp + c);
                ss += v.x; ss += v.y; ss += v.z; ss += v.w;
            }
        } else {
            for (int c = 0; c < nchunk; ++c) ss += rp[c];
        }
        sn += static_cast<double>(sqrtf(ss));
    }
    sp = wave_sum(sp);
    sn = wave_sum(sn);
    if (lane == 0) { red[0][wave] = sp; red[1][wave] = sn; }
    __syncthreads();
    if (threadIdx.x == 0) {
        double tp = 0.0, tn = 0.0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) { tp += red[0][w]; tn += red[1][w]; }
        n[e] += cnt;
        p_total[e] = static_cast<float>(static_cast<double>(p_total[e]) + tp);
        const double a = static_cast<double>(alpha);
        c_s[e] = static_cast<float>((1.0 - a) * static_cast<double>(c_s[e]) + a * (tn / cnt));
    }
}

__global__ __launch_bounds__(kThreads) void update_accounts_kernel(AccountJob j) { account_update(j, blockIdx.x); }

// One workgroup per token row of d <= kMixMax elements: v = the row's
// split partials added in split order (or the bf16 source row), h = bf16(v)
// (written when h_out is set), then u = bf16(h * (1 / sqrt(mean(h^2) + eps)))
// with the sum of squares taken over the bf16 values, per thread then per
// wave (butterfly) then over the waves in order.
// S = the number of split partials (a template argument, so that every
// slice's load is issued before the first add; 0 = read the bf16 source row).
constexpr int kMixVec = 4;                                  // floats per thread and group
constexpr int kMixGroups = 8;                               // d <= 256 * 4 * 8 = 8192
// Workgroups past the T rows do the deferred account update, one expert each.
template <int S>
__global__ __launch_bounds__(kThreads) void mix_norm_kernel(const float* __restrict__ part, int64_t split_stride,
                                                            const uint16_t* __restrict__ src, int T, int d, float eps,
                                                            uint16_t* __restrict__ h_out, uint16_t* __restrict__ u_out,
                                                            AccountJob job) {
    __shared__ float red[kWaves];
    const int t = blockIdx.x;
    if (t >= T) {                             // uniform over the workgroup
        account_update(job, t - T);
        return;
    }
    const int lane = lane_id(), wave = threadIdx.x / kWave;
    float v[kMixGroups][kMixVec];
    float ss = 0.f;
#pragma unroll
    for (int g = 0; g < kMixGroups; ++g) {
        const int j = (g * kThreads + threadIdx.x) * kMixVec;
        if (j >= d) continue;
        const size_t o = static_cast<size_t>(t) * d + j;
        if constexpr (S > 0) {
            float4 r[S];
#pragma unroll
            for (int sp = 0; sp < S; ++sp) r[sp] = *reinterpret_cast<const float4*>(part + sp * split_stride + o);
            float4 q = r[0];
#pragma unroll
            for (int sp = 1; sp < S; ++sp) { q.x += r[sp].x; q.y += r[sp].y; q.z += r[sp].z; q.w += r[sp].w; }
            v[g][0] = bf16_to_f32(f32_to_bf16(q.x)); v[g][1] = bf16_to_f32(f32_to_bf16(q.y));
            v[g][2] = bf16_to_f32(f32_to_bf16(q.z)); v[g][3] = bf16_to_f32(f32_to_bf16(q.w));
        } else {
            const uint2 q = *reinterpret_cast<const uint2*>(src + o);
            v[g][0] = bf16_to_f32(static_cast<uint16_t>(q.x & 0xffffu));
            v[g][1] = bf16_to_f32(static_cast<uint16_t>(q.x >> 16));
            v[g][2] = bf16_to_f32(static_cast<uint16_t>(q.y & 0xffffu));
            v[g][3] = bf16_to_f32(static_cast<uint16_t>(q.y >> 16));
        }
#pragma unroll
        for (int i = 0; i < kMixVec; ++i) ss = fmaf(v[g][i], v[g][i], ss);
        if (h_out) {
            uint2 pk;
            pk.x = static_cast<uint32_t>(f32_to_bf16(v[g][0])) | (static_cast<uint32_t>(f32_to_bf16(v[g][1])) << 16);
            pk.y = static_cast<uint32_t>(f32_to_bf16(v[g][2])) | (static_cast<uint32_t>(f32_to_bf16(v[g][3])) << 16);
            *reinterpret_cast<uint2*>(h_out + o) = pk;
        }
    }
    if (!u_out) return;
    ss = wave_sum(ss);
    if (lane == 0) red[wave] = ss;
    __syncthreads();
    float tot = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) tot += red[w];
    const float scale = 1.0f / sqrtf(tot / static_cast<float>(d) + eps);
#pragma unroll
    for (int g = 0; g < kMixGroups; ++g) {
        const int j = (g * kThreads + threadIdx.x) * kMixVec;
        if (j >= d) continue;
        uint2 pk;
        pk.x = static_cast<uint32_t>(f32_to_bf16(v[g][0] * scale)) |
               (static_cast<uint32_t>(f32_to_bf16(v[g][1] * scale)) << 16);
        pk.y = static_cast<uint32_t>(f32_to_bf16(v[g][2] * scale)) |
               (static_cast<uint32_t>(f32_to_bf16(v[g][3] * scale)) << 16);
        *reinterpret_cast<uint2*>(u_out + static_cast<size_t>(t) * d + j) = pk;
    }
}

// One thread per expert, grid-stride, so every one of the E <= kMaxExperts
// entries is cleared whatever the launch shape.
__global__ __launch_bounds__(kThreads) void reset_accounts_kernel(int E, int64_t* n, float* p, float* c) {
    for (int e = blockIdx.x * kThreads + threadIdx.x; e < E; e += gridDim.x * kThreads) {
        n[e] = 0;
        p[e] = 0.f;
        c[e] = 0.f;
    }
}

}  // namespace

int combine_chunks(const eat_params_t& p) { return (p.d_model / 4 + kThreads - 1) / kThreads; }

hipError_t launch_combine(const eat_params_t& p, int32_t T, const uint64_t* mask, const float* gate,
                          const int32_t* inv, const void* yp, const float* ys, const uint16_t* residual,
                          void* y, float* nrm2, int splits, int64_t split_stride, const int32_t* splits_dev,
                          bool rows_bf16, hipStream_t s) {
    if (splits < 1 || splits > kMaxSplits) return hipErrorInvalidValue;
    if (rows_bf16 && (splits != 1 || splits_dev || p.act_dtype != EAT_BF16)) return hipErrorInvalidValue;
    const int nchunk = combine_chunks(p);
    CombineArgs a{};
    a.mask = mask; a.gate = gate; a.inv = inv; a.yp = yp; a.splits_dev = splits_dev; a.ys = ys; a.res = residual;
    a.y = y; a.nrm2 = nrm2; a.split_stride = split_stride; a.splits = splits; a.T = T; a.E = p.E; a.d = p.d_model;
    a.nchunk = nchunk; a.words = mask_words(p.E);
    if (rows_bf16) {
        const int n8 = (p.d_model / kRowVec + kThreads - 1) / kThreads;
        combine_rows16_kernel<<<dim3(T, n8), kThreads, 0, s>>>(a);
        return hipGetLastError();
    }
    const dim3 grid(T, nchunk);
    if (p.act_dtype == EAT_BF16) combine_kernel<uint16_t><<<grid, kThreads, 0, s>>>(a);
    else combine_kernel<float><<<grid, kThreads, 0, s>>>(a);
    return hipGetLastError();
}

hipError_t launch_update_accounts(const eat_params_t& p, const int32_t* offsets, const int32_t* tok_idx,
                                  const float* prob, const float* nrm2, int parts, eat_accounts_t acc, hipStream_t s) {
    update_accounts_kernel<<<p.E, kThreads, 0, s>>>(AccountJob{offsets, tok_idx, prob, nrm2, parts, p.E, p.alpha, acc});
    return hipGetLastError();
}

bool mix_norm_fits(int d) { return d % (kMixVec * 2) == 0 && d <= kThreads * kMixVec * kMixGroups; }

hipError_t launch_mix_norm(const float* part, int splits, int64_t split_stride, const uint16_t* src, int32_t T,
                           int d, float eps, uint16_t* h_out, uint16_t* u_out, const AccountJob* accounts,
                           hipStream_t s) {
    const AccountJob job = accounts ? *accounts : AccountJob{};
    const int grid = T + job.experts;
    switch (splits) {
        case 0: mix_norm_kernel<0><<<grid, kThreads, 0, s>>>(part, split_stride, src, T, d, eps, h_out, u_out, job); break;
        case 1: mix_norm_kernel<1><<<grid, kThreads, 0, s>>>(part, split_stride, src, T, d, eps, h_out, u_out, job); break;
        case 2: mix_norm_kernel<2><<<grid, kThreads, 0, s>>>(part, split_stride, src, T, d, eps, h_out, u_out, job); break;
        case 4: mix_norm_kernel<4><<<grid, kThreads, 0, s>>>(part, split_stride, src, T, d, eps, h_out, u_out, job); break;
        case 8: mix_norm_kernel<8><<<grid, kThreads, 0, s>>>(part, split_stride, src, T, d, eps, h_out, u_out, job); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_reset_accounts(const eat_params_t& p, eat_accounts_t acc, hipStream_t s) {
    reset_accounts_kernel<<<(p.E + kThreads - 1) / kThreads, kThreads, 0, s>>>(p.E, acc.n, acc.p_total, acc.c_s);
    return hipGetLastError();
}

}  // namespace eat
