// Router + EAT selection kernel (gfx950).
//
// One workgroup of 16 waves routes a tile of 16 tokens:
//   1. history score S_h for every expert from the account snapshot
//      (Sec. 3.2, Eq. 1), in fp64, once per workgroup;
//   2. router logits for the 16 tokens x E experts with fp32 MFMA
//      (v_mfma_f32_16x16x4_f32); the 16 waves take interleaved 16-wide
//      k-steps of d and their partial tiles are added in wave order;
//   3. one wave per token, one lane per expert: softmax (Sec. 3.1), then
//      the mode's selection (EAT: Eq. 2-6 and Sec. 3.3; Top-K; Top-P) and
//      the renormalisation of Eq. 7-8.
// All reductions use fixed butterfly or sequential orders, so results are
// bit-reproducible run to run.
#include <math.h>

#include "eat_device.h"
#include "eat_internal.h"

namespace eat {
namespace {

constexpr int kTok = 16;            // tokens per workgroup
constexpr int kWaves = 16;

struct RouteArgs {
    const void* x;
    const float* w_router;
    const int64_t* acc_n;
    const float* acc_p;
    const float* acc_c;
    const int8_t* trend;
    uint64_t* mask;
    int32_t* k;
    float* gate;
    float* prob;
    int T, d, E, K, mode, cs_mode, top_p_cap;
    float top_p, w1, w2, w3, beta, alpha1, alpha2, kappa1, kappa2, ppl_up, ppl_down, q_lo, q_hi,
        eps, inv_temp;
};

template <typename XT>
__device__ __forceinline__ void load_x4(const XT* row, int k, float (&v)[4]);

template <>
__device__ __forceinline__ void load_x4<float>(const float* row, int k, float (&v)[4]) {
    const float4 q = *reinterpret_cast<const float4*>(row + k);
    v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
}
template <>
__device__ __forceinline__ void load_x4<uint16_t>(const uint16_t* row, int k, float (&v)[4]) {
    const uint2 q = *reinterpret_cast<const uint2*>(row + k);
    v[0] = __uint_as_float(q.x << 16);
    v[1] = __uint_as_float(q.x & 0xffff0000u);
    v[2] = __uint_as_float(q.y << 16);
    v[3] = __uint_as_float(q.y & 0xffff0000u);
}

// Value held by the lane whose rank (a permutation of 0..E-1) equals r.
__device__ __forceinline__ float value_at_rank(float v, int rank, int r, bool valid) {
    const uint64_t b = ballot(valid && rank == r);
    return read_lane(v, __builtin_ctzll(b));
}

template <typename XT, int NT>
__global__ __launch_bounds__(1024) void route_kernel(RouteArgs a) {
    __shared__ float part[kWaves][kTok][NT * 16];
    __shared__ float sh[64];

    const int lane = lane_id();
    const int wave = threadIdx.x / kWave;
    const int t0 = blockIdx.x * kTok;
    const int E = a.E;

    // ---- 1. history score from the account snapshot (Eq. 1) ----------
    if (a.mode == EAT_MODE_EAT && wave == 0) {
        const bool valid = lane < E;
        const double n = valid ? static_cast<double>(a.acc_n[lane]) : 0.0;
        const double pt = valid ? static_cast<double>(a.acc_p[lane]) : 0.0;
        const double c = valid ? static_cast<double>(a.acc_c[lane]) : 0.0;
        const double sum_n = wave_sum(n);
        const double t1 = sum_n > 0.0 ? n / sum_n : 0.0;
        const double t2 = n > 0.0 ? pt / n : 0.0;
        double t3 = c;
        if (a.cs_mode == 1) {
            const double sum_c = wave_sum(c);
            t3 = sum_c > 0.0 ? c / sum_c : 0.0;
        }
        sh[lane] = static_cast<float>(a.w1 * t1 + a.w2 * t2 + a.w3 * t3);
    }

    // ---- 2. router logits: MFMA 16 tokens x 16 experts x 4 k -----------
    {
        const XT* x = static_cast<const XT*>(a.x);
        const int row = t0 + (lane & 15);
        const bool row_ok = row < a.T;
        const XT* xrow = x + static_cast<size_t>(row_ok ? row : 0) * a.d;
        const int kq = 4 * (lane >> 4);        // this lane's 4 k values in a 16-k group
        const int nsteps = a.d / 16;            // 16-wide k-steps, dealt round-robin to the waves
        f32x4 acc[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        const float* wrow[NT];
        bool e_ok[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            const int e = nt * 16 + (lane & 15);
            e_ok[nt] = e < E;
            wrow[nt] = a.w_router + static_cast<size_t>(e_ok[nt] ? e : 0) * a.d;
        }
        auto step = [&](const float (&xv)[4], const float4 (&wv)[NT]) __attribute__((always_inline)) {
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                acc[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[0], wv[nt].x, acc[nt], 0, 0, 0);
                acc[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[1], wv[nt].y, acc[nt], 0, 0, 0);
                acc[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[2], wv[nt].z, acc[nt], 0, 0, 0);
                acc[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[3], wv[nt].w, acc[nt], 0, 0, 0);
            }
        };
        auto load = [&](int k, float (&xv)[4], float4 (&wv)[NT]) __attribute__((always_inline)) {
            xv[0] = xv[1] = xv[2] = xv[3] = 0.f;
            if (row_ok) load_x4<XT>(xrow, k + kq, xv);
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
                wv[nt] = e_ok[nt] ? *reinterpret_cast<const float4*>(wrow[nt] + k + kq)
                                  : make_float4(0.f, 0.f, 0.f, 0.f);
        };
        // groups of 4 of this wave's k-steps: loads first, then the MFMAs
        int st = wave;
        for (; st + 3 * kWaves < nsteps; st += 4 * kWaves) {
            float xv[4][4];
            float4 wv[4][NT];
#pragma unroll
            for (int u = 0; u < 4; ++u) load(16 * (st + u * kWaves), xv[u], wv[u]);
#pragma unroll
            for (int u = 0; u < 4; ++u) step(xv[u], wv[u]);
        }
        for (; st < nsteps; st += kWaves) {
            float xv[4];
            float4 wv[NT];
            load(16 * st, xv, wv);
            step(xv, wv);
        }
        // result layout: lane holds tokens 4*(lane/16)+i, expert nt*16 + lane%16
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int i = 0; i < 4; ++i) part[wave][4 * (lane >> 4) + i][nt * 16 + (lane & 15)] = acc[nt][i];
    }
    __syncthreads();

    // ---- 3. per-token softmax, selection, renormalisation --------------
    const bool valid = lane < E;
    for (int tl = wave; tl < kTok; tl += kWaves) {
        const int t = t0 + tl;
        if (t >= a.T) break;
        float z = -INFINITY;
        if (valid) {
            float sum = 0.f;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) sum += part[w][tl][lane];
            z = sum * a.inv_temp;
        }
        const float zmax = wave_max(z);
        const float ez = valid ? expf(z - zmax) : 0.f;
        const float p = ez / wave_sum(ez);

        uint64_t msk = 0;
        if (a.mode == EAT_MODE_EAT) {
            // Eq. 3-5 grounding on the token's routing weights
            const float mu = wave_sum(valid ? p : 0.f) / static_cast<float>(E);
            const float dv = valid ? p - mu : 0.f;
            const float sigma = sqrtf(wave_sum(dv * dv) / static_cast<float>(E));
            const float tau = fmaxf(a.alpha1 * mu, mu - a.alpha2 * sigma);
            // perplexity adjustment and smoothing (Sec. 3.3)
            const float f = (a.trend != nullptr && a.trend[t] > 0) ? a.ppl_up : a.ppl_down;
            const float tau_s = a.kappa1 * (f * tau) + a.kappa2 * tau;
            // bounds: q_lo / q_hi points of the sorted routing weights
            int rank = 0;
            for (int j = 0; j < E; ++j) {
                const float pj = read_lane(p, j);
                rank += (pj < p) || (pj == p && j < lane);
            }
            float qv[2];
            const float qs[2] = {a.q_lo, a.q_hi};
#pragma unroll
            for (int qi = 0; qi < 2; ++qi) {
                const float h = qs[qi] * static_cast<float>(E - 1);
                const int lo = static_cast<int>(floorf(h));
                const int hi = lo + 1 < E ? lo + 1 : E - 1;
                const float vlo = value_at_rank(p, rank, lo, valid);
                const float vhi = value_at_rank(p, rank, hi, valid);
                qv[qi] = vlo + (h - static_cast<float>(lo)) * (vhi - vlo);
            }
            const float tau_final = fminf(fmaxf(tau_s, qv[0]), qv[1]);
            // Eq. 2 importance and Eq. 6 activation set
            const float I = (1.f - a.beta) * p + a.beta * (valid ? sh[lane] : 0.f);
            const uint64_t cand = ballot(valid && I > tau_final);
            const int c = __popcll(cand);
            if (c == 0) {
                const float imax = wave_max(valid ? I : -INFINITY);
                const uint64_t b = ballot(valid && I == imax);
                msk = b & (~b + 1);                  // lowest index among maximisers
            } else if (c <= a.K) {
                msk = cand;
            } else {
                int beaten = 0;
                for (uint64_t rest = cand; rest; rest &= rest - 1) {
                    const int j = __builtin_ctzll(rest);
                    beaten += read_lane(I, j) > I;
                }
                msk = ballot(valid && ((cand >> lane) & 1ull) && beaten < a.K);
            }
        } else {
            // descending rank, ties to the lower expert index
            int rank = 0;
            for (int j = 0; j < E; ++j) {
                const float pj = read_lane(p, j);
                rank += (pj > p) || (pj == p && j < lane);
            }
            int kk;
            if (a.mode == EAT_MODE_TOPK) {
                kk = a.K;
            } else {
                // Top-P: shortest descending prefix whose running sum reaches top_p
                float run = 0.f;
                kk = E;
                for (int r = 0; r < E; ++r) {
                    run += value_at_rank(p, rank, r, valid);
                    if (run >= a.top_p) { kk = r + 1; break; }
                }
                if (a.top_p_cap > 0 && kk > a.top_p_cap) kk = a.top_p_cap;
            }
            msk = ballot(valid && rank < kk);
            // Ranks are a permutation for ordered values; NaN scores would
            // break that, so never keep more than kk experts (the workspace
            // holds at most kk rows per token in these modes).
            if (__popcll(msk) > kk) {
                uint64_t keep = 0, rest = msk;
                for (int i = 0; i < kk; ++i) { keep |= rest & (~rest + 1); rest &= rest - 1; }
                msk = keep;
            }
        }
        // Eq. 7-8 renormalisation over the selected experts
        const bool on = valid && ((msk >> lane) & 1ull);
        const float g = on ? p : 0.f;
        const float gsum = wave_sum(g);
        if (valid) {
            a.gate[static_cast<size_t>(t) * E + lane] = g / (gsum + a.eps);
            if (a.prob) a.prob[static_cast<size_t>(t) * E + lane] = p;
        }
        if (lane == 0) {
            a.mask[t] = msk;
            a.k[t] = __popcll(msk);
        }
    }
}

template <typename XT>
hipError_t launch_route_t(const RouteArgs& a, hipStream_t s) {
    const dim3 grid((a.T + kTok - 1) / kTok), block(kWaves * kWave);
    static_assert(kTok == kWaves, "one selection wave per token of the tile");
    const int nt = (a.E + 15) / 16;
    switch (nt) {
        case 1: route_kernel<XT, 1><<<grid, block, 0, s>>>(a); break;
        case 2: route_kernel<XT, 2><<<grid, block, 0, s>>>(a); break;
        case 3: route_kernel<XT, 3><<<grid, block, 0, s>>>(a); break;
        default: route_kernel<XT, 4><<<grid, block, 0, s>>>(a); break;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_route(const eat_params_t& p, const void* x, int32_t T, const float* w_router,
                        eat_accounts_t acc, const int8_t* trend, uint64_t* mask, int32_t* k,
                        float* gate, float* prob, hipStream_t s) {
    RouteArgs a;
    a.x = x; a.w_router = w_router;
    a.acc_n = acc.n; a.acc_p = acc.p_total; a.acc_c = acc.c_s;
    a.trend = trend; a.mask = mask; a.k = k; a.gate = gate; a.prob = prob;
    a.T = T; a.d = p.d_model; a.E = p.E; a.K = p.top_k; a.mode = p.mode; a.cs_mode = p.cs_mode;
    a.top_p_cap = p.top_p_cap; a.top_p = p.top_p;
    a.w1 = p.w1; a.w2 = p.w2; a.w3 = p.w3; a.beta = p.beta; a.alpha1 = p.alpha1; a.alpha2 = p.alpha2;
    a.kappa1 = p.kappa1; a.kappa2 = p.kappa2; a.ppl_up = p.ppl_up; a.ppl_down = p.ppl_down;
    a.q_lo = p.q_lo; a.q_hi = p.q_hi; a.eps = p.eps; a.inv_temp = p.inv_temperature;
    if (p.act_dtype == EAT_BF16) return launch_route_t<uint16_t>(a, s);
    return launch_route_t<float>(a, s);
}

}  // namespace eat
