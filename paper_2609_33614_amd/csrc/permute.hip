// Token -> expert permutation (gfx950).
//
// The selected (token, expert) pairs are laid out expert-major: expert e
// owns rows [offsets[e], offsets[e+1]), and inside that range its tokens
// appear in increasing token order.  One workgroup per expert:
//   offsets[e] = sum_t popcount(mask_t & bits below e)
// (a token's mask is W = ceil(E / 64) words; expert e is bit e % 64 of word
// e / 64, so the words before e's word count whole)
// needs no global histogram, so no inter-workgroup synchronisation or
// atomics.  Positions inside the segment come from wave ballots and an
// LDS-staged prefix over the 4 waves, chunk by chunk in token order.
#include "eat_device.h"
#include "eat_internal.h"

namespace eat {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;

// PRE: chunks of kThreads tokens whose mask words are loaded together (1
// for calls of at most kThreads tokens, where more would only add loads).
template <int PRE>
__global__ __launch_bounds__(kThreads) void permute_kernel(
    const uint64_t* __restrict__ mask, int T, int E, int W, int32_t* __restrict__ offsets,
    int32_t* __restrict__ tok_idx, int32_t* __restrict__ inv, int32_t* __restrict__ row_expert,
    int32_t* __restrict__ expert_load) {
    __shared__ int red[2][kWaves];
    __shared__ int wtot[kWaves];
    const int e = blockIdx.x;
    const int lane = lane_id(), wave = threadIdx.x / kWave;
    const int we = e >> 6, be = e & 63;
    const uint64_t below = (be == 0) ? 0ull : ((~0ull) >> (64 - be));
    const uint64_t bit = 1ull << be;

    // Both passes walk the tokens kPre chunks of kThreads at a time, loading
    // the chunks' mask words before using any (one memory round trip per
    // kPre chunks, not per chunk; tokens past T read token 0's word and are
    // off).
    constexpr int kPre = PRE;
    auto load_words = [&](int base0, int word, uint64_t (&mw)[kPre]) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < kPre; ++i) {
            const int t = base0 + i * kThreads + static_cast<int>(threadIdx.x);
            mw[i] = mask[static_cast<size_t>(t < T ? t : 0) * W + word];
        }
    };

    // segment start and size
    int before = 0, mine = 0;
    for (int base0 = 0; base0 < T; base0 += kPre * kThreads) {
        uint64_t mw[kPre];
        load_words(base0, we, mw);
#pragma unroll
        for (int i = 0; i < kPre; ++i) {
            const bool in = base0 + i * kThreads + static_cast<int>(threadIdx.x) < T;
            before += in ? __popcll(mw[i] & below) : 0;
            mine += (in && (mw[i] & bit)) ? 1 : 0;
        }
        for (int w = 0; w < we; ++w) {        // the whole words of lower experts (E > 64)
            load_words(base0, w, mw);
#pragma unroll
            for (int i = 0; i < kPre; ++i)
                before += base0 + i * kThreads + static_cast<int>(threadIdx.x) < T ? __popcll(mw[i]) : 0;
        }
    }
    before = wave_sum(before);
    mine = wave_sum(mine);
    if (lane == 0) { red[0][wave] = before; red[1][wave] = mine; }
    __syncthreads();
    int off = 0, cnt = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) { off += red[0][w]; cnt += red[1][w]; }
    if (threadIdx.x == 0) {
        offsets[e] = off;
        if (e == E - 1) offsets[E] = off + cnt;
        if (expert_load) expert_load[e] = cnt;
    }

    // ordered scatter of this expert's tokens
    int running = 0;
    const uint64_t lt = (lane == 0) ? 0ull : ((~0ull) >> (64 - lane));
    for (int base0 = 0; base0 < T; base0 += kPre * kThreads) {
        uint64_t mw[kPre];
        load_words(base0, we, mw);
#pragma unroll
        for (int i = 0; i < kPre; ++i) {
            const int base = base0 + i * kThreads;
            if (base >= T) break;             // uniform
            const int t = base + threadIdx.x;
            const bool on = t < T && (mw[i] & bit);
            const uint64_t b = ballot(on);
            if (lane == 0) wtot[wave] = __popcll(b);
            __syncthreads();
            int pre = 0, all = 0;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) {
                pre += (w < wave) ? wtot[w] : 0;
                all += wtot[w];
            }
            if (on) {
                const int row = off + running + pre + __popcll(b & lt);
                tok_idx[row] = t;
                row_expert[row] = e;
                inv[static_cast<size_t>(t) * E + e] = row;
            }
            running += all;
            __syncthreads();
        }
    }
}

}  // namespace

hipError_t launch_permute(const eat_params_t& p, int32_t T, const uint64_t* mask, int32_t* offsets,
                          int32_t* tok_idx, int32_t* inv, int32_t* row_expert, int32_t* expert_load,
                          hipStream_t s) {
    if (T <= kThreads)
        permute_kernel<1><<<dim3(p.E), dim3(kThreads), 0, s>>>(mask, T, p.E, mask_words(p.E), offsets, tok_idx,
                                                               inv, row_expert, expert_load);
    else
        permute_kernel<16><<<dim3(p.E), dim3(kThreads), 0, s>>>(mask, T, p.E, mask_words(p.E), offsets, tok_idx,
                                                                inv, row_expert, expert_load);
    return hipGetLastError();
}

}  // namespace eat
