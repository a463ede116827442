// Router + EAT selection kernels (gfx950).
//
// logits_kernel: one workgroup of 4 waves per (tile of 16*TT tokens,
// slice of d, group of 64 experts).  Router scores x W_r^T for the tile's
// tokens and the group's experts over its slice, fp32 MFMA
// (v_mfma_f32_16x16x4_f32, fp32 router weights); the waves take interleaved
// 16-wide k-steps of the slice and add their tiles in wave order; the
// slice's partial scores go to the workspace.  Spreading d over many
// workgroups keeps the router-weight reads (E*d*4 bytes per token tile) off
// a single CU.
//
// select_kernel<J>: one wave per token; lane l holds experts l, 64 + l, ...
// (J = ceil(E / 64) of them), and the token's mask is J 64-bit words, word
// j being the wave ballot over experts 64 j .. 64 j + 63.  Adds the slice
// partials in slice order, then softmax (Sec. 3.1), the optional OPD
// reweighting (Sec. 3.5) and the mode's selection
// (EAT: history score S_h from the account snapshot in fp64 (Eq. 1),
// importance (Eq. 2), threshold (Eq. 3-5, Sec. 3.3), activation set (Eq. 6);
// Top-K; Top-P) and the renormalisation of Eq. 7-8.  Orderings over a
// token's experts (the quantile bounds' ranks, Top-K / Top-P ranks, the
// candidates that beat a candidate) are counts against the other lanes'
// values, read back from LDS as broadcasts.
// All reductions use fixed butterfly or sequential orders, so results are
// bit-reproducible run to run.
#include <math.h>

#include <algorithm>

#include "eat_device.h"
#include "eat_internal.h"

namespace eat {
namespace {

constexpr int kLogitWaves = 4;
constexpr int kMaxRouteSlices = 16;     // d slices of the router scores

struct RouteArgs {
    const void* x;
    const float* w_router;
    const int64_t* acc_n;
    const float* acc_p;
    const float* acc_c;
    const int8_t* trend;
    float* part;               // [slices][T][E] partial router scores
    uint64_t* mask;            // [T][J] words
    int32_t* k;
    float* gate;
    float* prob;
    const float* scale;        // OPD per-expert reweighting [E], or null
    int T, d, E, K, mode, cs_mode, top_p_cap, slices;
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

// Value of the expert whose rank (a permutation of 0..E-1 for ordered
// values) equals r; NaN when no expert holds it (NaN scores).
template <int J>
__device__ __forceinline__ float value_at_rank(const float (&v)[J], const int (&rank)[J], int r,
                                               const bool (&valid)[J]) {
    float out = NAN;
    bool found = false;
#pragma unroll
    for (int j = 0; j < J; ++j) {
        const uint64_t b = ballot(valid[j] && rank[j] == r);
        if (!found && b) {
            out = read_lane(v[j], __builtin_ctzll(b));
            found = true;
        }
    }
    return out;
}

typedef uint64_t u64x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Lanes of one wave exchanging values through LDS: every lane's stores are
// ordered before the loads that follow (a wave's LDS operations run in
// issue order; the fences keep the compiler from moving them).
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Order-preserving bits of a non-NaN float: a < b exactly when
// ord_bits(a) < ord_bits(b); -0 and +0 (equal values) map alike.
__device__ __forceinline__ uint32_t ord_bits(float f) {
    const uint32_t u = f == 0.f ? 0u : __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Ranks of a token's E values (lane l of group j holds expert 64 j + l):
// how many values come before each one, ascending (ASC) or descending, with
// equal values in expert-index order, so the ranks are a permutation of
// 0..E-1.  Only for values without NaN.  Each value becomes one 64-bit key
// (order-preserving bits, then the expert index); the wave's keys go to
// `kbuf` (this wave's 64 J LDS entries, 16-byte aligned), and every lane
// counts the keys below its own, reading them two at a time from one address
// for the whole wave (a broadcast: two compares per value, against a lane
// read and three hazard-separated scalar steps per value for the readlane
// loop).  `srt` (64 J floats of LDS) receives the values in rank order.
template <int J, bool ASC>
__device__ __forceinline__ void rank_by_keys(const float (&v)[J], const bool (&valid)[J], int E,
                                             uint64_t* kbuf, float* srt, int (&rank)[J]) {
    const int lane = lane_id();
    uint64_t key[J];
#pragma unroll
    for (int j = 0; j < J; ++j) {
        const uint32_t o = ASC ? ord_bits(v[j]) : ~ord_bits(v[j]);
        key[j] = valid[j] ? (static_cast<uint64_t>(o) << 32) | static_cast<uint32_t>(64 * j + lane) : ~0ull;
        kbuf[64 * j + lane] = key[j];
        rank[j] = 0;
    }
    wave_lds_sync();
    // an odd E reads one entry past it: an all-ones key, below no key
    for (int l = 0; l < E; l += 2) {
        const u64x2 q = *reinterpret_cast<const u64x2*>(kbuf + l);
#pragma unroll
        for (int j = 0; j < J; ++j) rank[j] += static_cast<int>(q.x < key[j]) + static_cast<int>(q.y < key[j]);
    }
#pragma unroll
    for (int j = 0; j < J; ++j)
        if (valid[j]) srt[rank[j]] = v[j];
    wave_lds_sync();
}

template <typename XT, int NT, int TT>
__global__ __launch_bounds__(256) void logits_kernel(RouteArgs a) {
    __shared__ float red[kLogitWaves][TT * 16][NT * 16];
    const int lane = lane_id();
    const int wave = threadIdx.x / kWave;
    const int t0 = blockIdx.x * 16 * TT;
    const int E = a.E;
    const int e0 = blockIdx.z * 64;              // this workgroup's expert group
    const int EG = min(64, E - e0);
    const XT* x = static_cast<const XT*>(a.x);
    const int kq = 4 * (lane >> 4);          // this lane's 4 k values in a 16-wide k-step
    const int nsteps = a.d / 16;
    const int per = nsteps / a.slices;
    const int sbeg = blockIdx.y * per, send = sbeg + per;

    const XT* xrow[TT];
    bool row_ok[TT];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
        const int row = t0 + tt * 16 + (lane & 15);
        row_ok[tt] = row < a.T;
        xrow[tt] = x + static_cast<size_t>(row_ok[tt] ? row : 0) * a.d;
    }
    const float* wrow[NT];
    bool e_ok[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        const int e = e0 + nt * 16 + (lane & 15);
        e_ok[nt] = e < E;
        wrow[nt] = a.w_router + static_cast<size_t>(e_ok[nt] ? e : 0) * a.d;
    }
    f32x4 acc[TT][NT];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[tt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Every load is unconditional: token rows past T and experts past E read
    // row 0, which exists, and their scores are never written.  (A load under
    // a per-lane branch makes the compiler wait for it inside the branch, one
    // round trip per group of k-steps.)
    auto load = [&](int k, float (&xv)[TT][4], float4 (&wv)[NT]) __attribute__((always_inline)) {
#pragma unroll
        for (int tt = 0; tt < TT; ++tt) load_x4<XT>(xrow[tt], k + kq, xv[tt]);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) wv[nt] = *reinterpret_cast<const float4*>(wrow[nt] + k + kq);
    };
    auto step = [&](const float (&xv)[TT][4], const float4 (&wv)[NT]) __attribute__((always_inline)) {
#pragma unroll
        for (int tt = 0; tt < TT; ++tt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                acc[tt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[tt][0], wv[nt].x, acc[tt][nt], 0, 0, 0);
                acc[tt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[tt][1], wv[nt].y, acc[tt][nt], 0, 0, 0);
                acc[tt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[tt][2], wv[nt].z, acc[tt][nt], 0, 0, 0);
                acc[tt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[tt][3], wv[nt].w, acc[tt][nt], 0, 0, 0);
            }
    };
    // groups of G of this wave's k-steps: all loads of a group, then its MFMAs
    constexpr int G = TT * NT <= 2 ? 4 : 2;
    int st = sbeg + wave;
    for (; st + (G - 1) * kLogitWaves < send; st += G * kLogitWaves) {
        float xv[G][TT][4];
        float4 wv[G][NT];
#pragma unroll
        for (int u = 0; u < G; ++u) load(16 * (st + u * kLogitWaves), xv[u], wv[u]);
#pragma unroll
        for (int u = 0; u < G; ++u) step(xv[u], wv[u]);
    }
    for (; st < send; st += kLogitWaves) {
        float xv[TT][4];
        float4 wv[NT];
        load(16 * st, xv, wv);
        step(xv, wv);
    }
    // lane holds tokens tt*16 + 4*(lane/16) + i, expert nt*16 + lane%16
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int i = 0; i < 4; ++i) red[wave][tt * 16 + 4 * (lane >> 4) + i][nt * 16 + (lane & 15)] = acc[tt][nt][i];
    __syncthreads();
    for (int v = threadIdx.x; v < TT * 16 * EG; v += 256) {
        const int tl = v / EG, e = v % EG;
        const int t = t0 + tl;
        if (t >= a.T) continue;
        float sum = 0.f;
#pragma unroll
        for (int w = 0; w < kLogitWaves; ++w) sum += red[w][tl][e];
        a.part[(static_cast<size_t>(blockIdx.y) * a.T + t) * E + e0 + e] = sum;
    }
}

constexpr int kSelWaves = 4;

// Sum over the wave of each lane's J values (lane-local first, in expert
// order, then the butterfly); for J = 1 this is the plain butterfly.
template <int J>
__device__ __forceinline__ float wave_sum_j(const float (&v)[J]) {
    float s = v[0];
#pragma unroll
    for (int j = 1; j < J; ++j) s += v[j];
    return wave_sum(s);
}

template <int J>
__global__ __launch_bounds__(256) void select_kernel(RouteArgs a) {
    __shared__ float sh[64 * J];
    __shared__ __align__(16) uint64_t kb[kSelWaves][64 * J];   // per-wave rank keys
    __shared__ __align__(16) float srt[kSelWaves][64 * J];     // per-wave values in rank order
    const int lane = lane_id();
    const int wave = threadIdx.x / kWave;
    const int E = a.E;
    bool valid[J];
#pragma unroll
    for (int j = 0; j < J; ++j) valid[j] = 64 * j + lane < E;

    // ---- this token's partial router scores: every slice's load issued
    // before the history score below, summed (in slice order) after it ----
    // The kernel's loads are all issued here, before any of them is waited
    // for, from clamped in-bounds addresses (token 0, expert 0, slice 0, or the
    // partial-score buffer standing in for an absent trend or scale); values
    // read for lanes past E or slices past the call's are never used.  (A load
    // under a per-lane branch makes the compiler wait for it inside the
    // branch, a round trip each.)
    const int t = blockIdx.x * kSelWaves + wave;
    const bool tok = t < a.T;
    const int tc = tok ? t : 0;
    float zp[J][kMaxRouteSlices];
#pragma unroll
    for (int j = 0; j < J; ++j) {
        const float* src = a.part + static_cast<size_t>(tc) * E + (valid[j] ? 64 * j + lane : 0);
        const size_t stride = static_cast<size_t>(a.T) * E;
#pragma unroll
        for (int sl = 0; sl < kMaxRouteSlices; ++sl) zp[j][sl] = src[(sl < a.slices ? sl : 0) * stride];
    }
    const int8_t trend_t = *(a.trend ? a.trend + tc : reinterpret_cast<const int8_t*>(a.part));
    float scale[J];
#pragma unroll
    for (int j = 0; j < J; ++j) scale[j] = (a.scale ? a.scale : a.part)[valid[j] ? 64 * j + lane : 0];

    // ---- history score from the account snapshot (Eq. 1) --------------
    if (a.mode == EAT_MODE_EAT && wave == 0) {
        double n[J], pt[J], c[J];
#pragma unroll
        for (int j = 0; j < J; ++j) {
            // relaxed loads: plain loads that the compiler does not move
            // under the lane test below (and then wait for one by one)
            const int e = valid[j] ? 64 * j + lane : 0;
            const int64_t nv = __hip_atomic_load(a.acc_n + e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            const float pv = __hip_atomic_load(a.acc_p + e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            const float cv = __hip_atomic_load(a.acc_c + e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            n[j] = valid[j] ? static_cast<double>(nv) : 0.0;
            pt[j] = valid[j] ? static_cast<double>(pv) : 0.0;
            c[j] = valid[j] ? static_cast<double>(cv) : 0.0;
        }
        double ln = n[0], lc = c[0];
#pragma unroll
        for (int j = 1; j < J; ++j) { ln += n[j]; lc += c[j]; }
        const double sum_n = wave_sum(ln);
        const double sum_c = a.cs_mode == 1 ? wave_sum(lc) : 0.0;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const double t1 = sum_n > 0.0 ? n[j] / sum_n : 0.0;
            const double t2 = n[j] > 0.0 ? pt[j] / n[j] : 0.0;
            double t3 = c[j];
            if (a.cs_mode == 1) t3 = sum_c > 0.0 ? c[j] / sum_c : 0.0;
            sh[64 * j + lane] = static_cast<float>(a.w1 * t1 + a.w2 * t2 + a.w3 * t3);
        }
    }
    __syncthreads();

    // ---- per-token softmax, selection, renormalisation ----------------
    if (!tok) return;
    float z[J];
#pragma unroll
    for (int j = 0; j < J; ++j) {
        float sum = 0.f;
#pragma unroll
        for (int sl = 0; sl < kMaxRouteSlices; ++sl)
            if (sl < a.slices) sum += zp[j][sl];
        z[j] = valid[j] ? sum * a.inv_temp : -INFINITY;
    }
    float zl = z[0];
#pragma unroll
    for (int j = 1; j < J; ++j) zl = fmaxf(zl, z[j]);
    const float zmax = wave_max(zl);
    float p[J];
#pragma unroll
    for (int j = 0; j < J; ++j) p[j] = valid[j] ? expf(z[j] - zmax) : 0.f;
    {
        const float den = wave_sum_j<J>(p);
#pragma unroll
        for (int j = 0; j < J; ++j) p[j] = p[j] / den;
    }
    if (a.scale) {
        // Sec. 3.5: OPD reweighting, p'_i = s_i p_i / sum_j s_j p_j, used for
        // everything below (importance, threshold, selection, gates, P_total)
#pragma unroll
        for (int j = 0; j < J; ++j) p[j] = valid[j] ? scale[j] * p[j] : 0.f;
        const float den = wave_sum_j<J>(p);
#pragma unroll
        for (int j = 0; j < J; ++j) p[j] = p[j] / den;
    }

    // Without NaN among the token's weights the ranks below come from LDS
    // keys; a token with NaN weights keeps the lane-by-lane comparisons, whose
    // treatment of NaN (it compares as neither smaller nor larger, so it
    // takes rank 0 and the ranks of the others close up) is the documented
    // rule for non-finite tokens.
    uint64_t nan_lanes = 0;
#pragma unroll
    for (int j = 0; j < J; ++j) nan_lanes |= ballot(valid[j] && p[j] != p[j]);
    const bool by_keys = nan_lanes == 0;
    uint64_t* const kbw = kb[wave];
    float* const srtw = srt[wave];

    uint64_t msk[J];
#pragma unroll
    for (int j = 0; j < J; ++j) msk[j] = 0;
    if (a.mode == EAT_MODE_EAT) {
        // Eq. 3-5 grounding on the token's routing weights
        float tmp[J];
#pragma unroll
        for (int j = 0; j < J; ++j) tmp[j] = valid[j] ? p[j] : 0.f;
        const float mu = wave_sum_j<J>(tmp) / static_cast<float>(E);
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const float dv = valid[j] ? p[j] - mu : 0.f;
            tmp[j] = dv * dv;
        }
        const float sigma = sqrtf(wave_sum_j<J>(tmp) / static_cast<float>(E));
        const float tau = fmaxf(a.alpha1 * mu, mu - a.alpha2 * sigma);
        // perplexity adjustment and smoothing (Sec. 3.3)
        const float f = (a.trend != nullptr && trend_t > 0) ? a.ppl_up : a.ppl_down;
        const float tau_s = a.kappa1 * (f * tau) + a.kappa2 * tau;
        // bounds: q_lo / q_hi points of the sorted routing weights
        int rank[J];
        if (by_keys) {
            rank_by_keys<J, true>(p, valid, E, kbw, srtw, rank);
        } else {
#pragma unroll
            for (int j = 0; j < J; ++j) rank[j] = 0;
#pragma unroll
            for (int jj = 0; jj < J; ++jj) {
                const int nl = min(64, E - 64 * jj);
                for (int l = 0; l < nl; ++l) {
                    const float pv = read_lane(p[jj], l);
                    const int ev = 64 * jj + l;
#pragma unroll
                    for (int j = 0; j < J; ++j) rank[j] += (pv < p[j]) || (pv == p[j] && ev < 64 * j + lane);
                }
            }
        }
        float qv[2];
        const float qs[2] = {a.q_lo, a.q_hi};
#pragma unroll
        for (int qi = 0; qi < 2; ++qi) {
            const float h = qs[qi] * static_cast<float>(E - 1);
            const int lo = static_cast<int>(floorf(h));
            const int hi = lo + 1 < E ? lo + 1 : E - 1;
            const float vlo = by_keys ? srtw[lo] : value_at_rank<J>(p, rank, lo, valid);
            const float vhi = by_keys ? srtw[hi] : value_at_rank<J>(p, rank, hi, valid);
            qv[qi] = vlo + (h - static_cast<float>(lo)) * (vhi - vlo);
        }
        const float tau_final = fminf(fmaxf(tau_s, qv[0]), qv[1]);
        // Eq. 2 importance and Eq. 6 activation set
        float I[J];
        uint64_t cand[J];
        int c = 0;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            I[j] = (1.f - a.beta) * p[j] + a.beta * (valid[j] ? sh[64 * j + lane] : 0.f);
            cand[j] = ballot(valid[j] && I[j] > tau_final);
            c += __popcll(cand[j]);
        }
        if (c == 0) {
            // argmax of I, lowest index among maximisers
            float il = -INFINITY;
#pragma unroll
            for (int j = 0; j < J; ++j) il = fmaxf(il, valid[j] ? I[j] : -INFINITY);
            const float imax = wave_max(il);
            bool done = false;
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const uint64_t b = ballot(valid[j] && I[j] == imax);
                if (!done && b) { msk[j] = b & (~b + 1); done = true; }
            }
        } else if (c <= a.K) {
#pragma unroll
            for (int j = 0; j < J; ++j) msk[j] = cand[j];
        } else {
            // keep the candidates beaten (strictly) by fewer than K others:
            // each lane counts the candidates' order-preserving importance
            // bits above its own (a candidate's importance exceeds the
            // threshold, so it is never NaN; other lanes store 0, below every
            // candidate's bits), four at a time from LDS broadcasts
            uint32_t* const ib = reinterpret_cast<uint32_t*>(kbw);
            uint32_t ki[J];
            int beaten[J];
#pragma unroll
            for (int j = 0; j < J; ++j) {
                ki[j] = ((cand[j] >> lane) & 1ull) ? ord_bits(I[j]) : 0u;
                ib[64 * j + lane] = ki[j];
                beaten[j] = 0;
            }
            wave_lds_sync();
            // entries up to E rounded to 4 hold 0 (lanes past E)
            for (int l = 0; l < E; l += 4) {
                const u32x4 q = *reinterpret_cast<const u32x4*>(ib + l);
#pragma unroll
                for (int j = 0; j < J; ++j)
                    beaten[j] += static_cast<int>(q.x > ki[j]) + static_cast<int>(q.y > ki[j]) +
                                 static_cast<int>(q.z > ki[j]) + static_cast<int>(q.w > ki[j]);
            }
#pragma unroll
            for (int j = 0; j < J; ++j) msk[j] = ballot(valid[j] && ((cand[j] >> lane) & 1ull) && beaten[j] < a.K);
        }
    } else {
        // descending rank, ties to the lower expert index
        int rank[J];
        if (by_keys) {
            rank_by_keys<J, false>(p, valid, E, kbw, srtw, rank);
        } else {
#pragma unroll
            for (int j = 0; j < J; ++j) rank[j] = 0;
#pragma unroll
            for (int jj = 0; jj < J; ++jj) {
                const int nl = min(64, E - 64 * jj);
                for (int l = 0; l < nl; ++l) {
                    const float pv = read_lane(p[jj], l);
                    const int ev = 64 * jj + l;
#pragma unroll
                    for (int j = 0; j < J; ++j) rank[j] += (pv > p[j]) || (pv == p[j] && ev < 64 * j + lane);
                }
            }
        }
        int kk;
        if (a.mode == EAT_MODE_TOPK) {
            kk = a.K;
        } else {
            // Top-P: shortest descending prefix whose running sum reaches top_p
            float run = 0.f;
            kk = E;
            for (int r = 0; r < E; ++r) {
                run += by_keys ? srtw[r] : value_at_rank<J>(p, rank, r, valid);
                if (run >= a.top_p) { kk = r + 1; break; }
            }
            if (a.top_p_cap > 0 && kk > a.top_p_cap) kk = a.top_p_cap;
        }
        int c = 0;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            msk[j] = ballot(valid[j] && rank[j] < kk);
            c += __popcll(msk[j]);
        }
        // Ranks are a permutation for ordered values; NaN scores would
        // break that, so never keep more than kk experts (the workspace
        // holds at most kk rows per token in these modes): the lowest
        // indices are kept.
        if (c > kk) {
            int left = kk;
#pragma unroll
            for (int j = 0; j < J; ++j) {
                uint64_t keep = 0, rest = msk[j];
                for (; left > 0 && rest; --left) { keep |= rest & (~rest + 1); rest &= rest - 1; }
                msk[j] = keep;
            }
        }
    }
    // Eq. 7-8 renormalisation over the selected experts
    float g[J];
    int kt = 0;
#pragma unroll
    for (int j = 0; j < J; ++j) {
        g[j] = (valid[j] && ((msk[j] >> lane) & 1ull)) ? p[j] : 0.f;
        kt += __popcll(msk[j]);
    }
    const float gsum = wave_sum_j<J>(g);
#pragma unroll
    for (int j = 0; j < J; ++j) {
        if (!valid[j]) continue;
        const size_t o = static_cast<size_t>(t) * E + 64 * j + lane;
        a.gate[o] = g[j] / (gsum + a.eps);
        if (a.prob) a.prob[o] = p[j];
    }
    if (lane == 0) {
#pragma unroll
        for (int j = 0; j < J; ++j) a.mask[static_cast<size_t>(t) * J + j] = msk[j];
        a.k[t] = kt;
    }
}

template <typename XT, int NT>
hipError_t launch_logits_n(const RouteArgs& a, int tt, dim3 grid, hipStream_t s) {
    if (tt == 4) logits_kernel<XT, NT, 4><<<grid, 256, 0, s>>>(a);
    else logits_kernel<XT, NT, 1><<<grid, 256, 0, s>>>(a);
    return hipGetLastError();
}

template <typename XT>
hipError_t launch_route_t(const RouteArgs& a, hipStream_t s) {
    const int tt = route_token_tiles(a.T);
    const int words = mask_words(a.E);
    const dim3 grid((a.T + 16 * tt - 1) / (16 * tt), a.slices, words);
    hipError_t err;
    switch ((std::min(a.E, 64) + 15) / 16) {
        case 1: err = launch_logits_n<XT, 1>(a, tt, grid, s); break;
        case 2: err = launch_logits_n<XT, 2>(a, tt, grid, s); break;
        case 3: err = launch_logits_n<XT, 3>(a, tt, grid, s); break;
        default: err = launch_logits_n<XT, 4>(a, tt, grid, s); break;
    }
    if (err != hipSuccess) return err;
    const dim3 sg((a.T + kSelWaves - 1) / kSelWaves), sb(kSelWaves * kWave);
    switch (words) {
        case 1: select_kernel<1><<<sg, sb, 0, s>>>(a); break;
        case 2: select_kernel<2><<<sg, sb, 0, s>>>(a); break;
        case 3: select_kernel<3><<<sg, sb, 0, s>>>(a); break;
        default: select_kernel<4><<<sg, sb, 0, s>>>(a); break;
    }
    return hipGetLastError();
}

}  // namespace

int route_token_tiles(int32_t T) { return T >= 1024 ? 4 : 1; }

int route_slices(const eat_params_t& p, int32_t T) {
    // enough (token tile, d slice) workgroups to spread the router weights
    // over the chip: about 512, each wave keeping at least one k-step, and
    // at most kMaxRouteSlices (the selection reads every slice of a score in
    // one round of loads)
    const int tiles = (T + 16 * route_token_tiles(T) - 1) / (16 * route_token_tiles(T));
    const int nsteps = p.d_model / 16;
    int sl = 1;
    while (2 * sl <= kMaxRouteSlices && 2 * sl * tiles <= 512 && nsteps % (2 * sl) == 0 &&
           nsteps / (2 * sl) >= kLogitWaves)
        sl *= 2;
    return sl;
}

hipError_t launch_route(const eat_params_t& p, const void* x, int32_t T, const float* w_router,
                        eat_accounts_t acc, const int8_t* trend, float* part, uint64_t* mask, int32_t* k,
                        float* gate, float* prob, hipStream_t s) {
    RouteArgs a;
    a.part = part;
    a.slices = route_slices(p, T);
    a.x = x; a.w_router = w_router;
    a.acc_n = acc.n; a.acc_p = acc.p_total; a.acc_c = acc.c_s;
    a.trend = trend; a.mask = mask; a.k = k; a.gate = gate; a.prob = prob;
    a.T = T; a.d = p.d_model; a.E = p.E; a.K = p.top_k; a.mode = p.mode; a.cs_mode = p.cs_mode;
    a.top_p_cap = p.top_p_cap; a.top_p = p.top_p;
    a.w1 = p.w1; a.w2 = p.w2; a.w3 = p.w3; a.beta = p.beta; a.alpha1 = p.alpha1; a.alpha2 = p.alpha2;
    a.kappa1 = p.kappa1; a.kappa2 = p.kappa2; a.ppl_up = p.ppl_up; a.ppl_down = p.ppl_down;
    a.q_lo = p.q_lo; a.q_hi = p.q_hi; a.eps = p.eps; a.inv_temp = p.inv_temperature;
    a.scale = p.expert_scale;
    if (p.act_dtype == EAT_BF16) return launch_route_t<uint16_t>(a, s);
    return launch_route_t<float>(a, s);
}

}  // namespace eat
