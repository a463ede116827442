// Expert FFN kernels (gfx950): SwiGLU experts over the expert-major rows.
//
//   up/gate:  H[r][f] = silu(x_t . W1_e[f]) * (x_t . W3_e[f])   t = tok_idx[r]
//   down:     Yp[r][j] = H[r] . W2_e[j]
//
// bf16 path ("stream" kernels): each wave owns 16 consecutive weight rows
// (the 16-row A operand of v_mfma_f32_16x16x32_bf16) and streams them over
// the whole reduction dimension once, applying them to up to 16*NSUB
// tokens of the same expert (the B operand, zero-padded).  Weight bytes are
// read from HBM exactly once per token tile, which is what bounds decode.
// Either projection may split its reduction dimension into slices, as many
// as the tiles in use call for (chosen on the device from the tile count,
// which only the device knows): the down projection's partial tiles are
// added, in split order, by the combine kernel; the up/gate projection's by
// a reduce kernel that then forms H = silu(G) * U.  (Adding them up inside
// the projection, by the last slice of a tile to finish, needs a device-wide
// release per work item, an L2 write-back on this part: measured slower.)
// The grid is persistent: a flat list of (token tile, slice, row block)
// work items over about as many workgroups as the chip keeps resident.
// Weights may be in the packed layout (pack.hip), read one contiguous
// kilobyte per load instruction with the streaming cache policy.
// Prefill-sized calls (hundreds of rows per expert) go to the wide MFMA
// tiles of wide.hip instead.
//
// fp32 path: plain dot products, one thread per output element, for layers
// whose weights are fp32 (small correctness-sized layers).
#include <algorithm>
#include <type_traits>

#include "eat_device.h"
#include "eat_internal.h"

namespace eat {
namespace {

// ---------------------------------------------------------------- fp32 --

struct F32Args {
    const float* x;            // [*, d] token activations
    const float* w1;           // [E][F][d]
    const float* w3;
    const float* w2;           // [E][d][F]
    const int32_t* tok_idx;    // row -> token, or null (row == token)
    const int32_t* row_expert; // row -> expert, or null (expert 0)
    const int32_t* rows_dev;   // device row count (offsets[E]), or null
    int rows_host;             // row count when rows_dev is null
    int d, F;
    float* h;                  // [rows][F]
    float* yp;                 // [rows][d]
};

__global__ __launch_bounds__(256) void ffn_up_f32(F32Args a) {
    const int64_t rows = a.rows_dev ? *a.rows_dev : a.rows_host;
    const int64_t total = rows * a.F;
    for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < total;
         i += int64_t(gridDim.x) * blockDim.x) {
        const int64_t r = i / a.F;
        const int f = static_cast<int>(i % a.F);
        const int t = a.tok_idx ? a.tok_idx[r] : static_cast<int>(r);
        const int e = a.row_expert ? a.row_expert[r] : 0;
        const float* xr = a.x + static_cast<size_t>(t) * a.d;
        const float* g = a.w1 + (static_cast<size_t>(e) * a.F + f) * a.d;
        const float* u = a.w3 + (static_cast<size_t>(e) * a.F + f) * a.d;
        float sg = 0.f, su = 0.f;
        for (int k = 0; k < a.d; ++k) {
            sg = fmaf(xr[k], g[k], sg);
            su = fmaf(xr[k], u[k], su);
        }
        a.h[r * a.F + f] = silu(sg) * su;
    }
}

__global__ __launch_bounds__(256) void ffn_down_f32(F32Args a) {
    const int64_t rows = a.rows_dev ? *a.rows_dev : a.rows_host;
    const int64_t total = rows * a.d;
    for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < total;
         i += int64_t(gridDim.x) * blockDim.x) {
        const int64_t r = i / a.d;
        const int j = static_cast<int>(i % a.d);
        const int e = a.row_expert ? a.row_expert[r] : 0;
        const float* hr = a.h + r * a.F;
        const float* w = a.w2 + (static_cast<size_t>(e) * a.d + j) * a.F;
        float s = 0.f;
        for (int f = 0; f < a.F; ++f) s = fmaf(hr[f], w[f], s);
        a.yp[r * a.d + j] = s;
    }
}

hipError_t launch_f32_pair(F32Args a, int64_t rows_cap, hipStream_t s,
                           const std::function<void()>& between) {
    const int64_t up = rows_cap * a.F, dn = rows_cap * a.d;
    const int gu = static_cast<int>(std::min<int64_t>((up + 255) / 256, 8192));
    const int gd = static_cast<int>(std::min<int64_t>((dn + 255) / 256, 8192));
    if (gu > 0) ffn_up_f32<<<gu, 256, 0, s>>>(a);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    if (between) between();
    if (gd > 0) ffn_down_f32<<<gd, 256, 0, s>>>(a);
    return hipGetLastError();
}

// ------------------------------------------------------- bf16 streaming --

// Reduction-dimension slices of a stream launch (split_rule): double them
// while the number of 16-row wave tiles over the token tiles in use is below
// a threshold.  The tiles in use (the experts a call's tokens touch) are
// only known on the device, so the kernel applies the rule itself; the host
// sizes the workspace for the most slices the rule can give.  Each slice
// costs one more fp32 row per assignment in the partial buffers.
#ifndef EAT_SPLIT_WAVES
#define EAT_SPLIT_WAVES 4096
#endif
// Once the grid holds ~1024 wave tiles, a slice keeps at least
// EAT_SPLIT_MIN_K reduction elements: shorter ones cost more in partial rows
// than their extra waves gain (measured: 4 slices of a 1024-wide down
// projection over 8 experts are slower than 2); smaller grids split down
// to 128 (the same projection over 2 experts gains from 4 slices).
#ifndef EAT_SPLIT_MIN_K
#define EAT_SPLIT_MIN_K 384
#endif
// The gated projection pays for its slices with fp32 G and U partials that a
// second kernel adds up (swiglu_reduce_kernel), so it only splits grids that
// would leave most of the chip idle.
#ifndef EAT_UP_SPLIT_WAVES
#define EAT_UP_SPLIT_WAVES 1024
#endif
// With 128-token tiles (calls of more than 64 tokens) an expert's tile is a
// small prefill, and up to 2048 waves pay: the fine-grained layer's 256-token
// EAT decode (~8 experts of ~256 tokens) +14%, Top-K unchanged; 1024 stays
// for smaller tiles (the Mixtral-shaped 64-token decode loses 10% at 2048).
#ifndef EAT_UP_SPLIT_WAVES_T128
#define EAT_UP_SPLIT_WAVES_T128 2048
#endif
#ifndef EAT_UP_SPLIT_MAX
#define EAT_UP_SPLIT_MAX 4
#endif

// The gated projection (gated = true) doubles only while the doubled count
// stays within the threshold, never past it: its slices cost fp32 G and U
// partials and a reduce launch, and a split that overshoots paid less than
// it cost (the 128-expert layer's EAT decode, ~15 experts of 64-token tiles
// around the 1024-wave threshold: +7% with it).  The plain projection keeps
// doubling until it reaches the threshold: the Mixtral-shaped down projection
// took 5% longer under the gated form.
__host__ __device__ inline int split_rule(int64_t rows_m, int kdim, int64_t tiles, int max_splits,
                                          int64_t threshold, bool gated) {
    const int64_t waves = (rows_m / 16) * tiles;
    int s = 1;
    while (s < max_splits && kdim % (64 * 2 * s) == 0 && (gated ? waves * s * 2 <= threshold : waves * s < threshold) &&
           kdim / (2 * s) >= (waves * s < 1024 ? 128 : EAT_SPLIT_MIN_K))
        s *= 2;
    return s;
}


struct StreamArgs {
    const uint16_t* wa;        // [groups][M][K]  (W1 for up/gate, W2 for down)
    const uint16_t* wb;        // [groups][M][K]  (W3, gated kernel only)
    const uint16_t* src;       // activation rows, K wide
    const int32_t* gather;     // row -> source row, or null (identity)
    const int32_t* offsets;    // [groups+1] expert-major row offsets, or null
    int nrows;                 // rows of the single group when offsets is null
    int groups, M, K;
    int splits;                // slices of the reduction dimension; with rule_threshold > 0
                               // the most the device-side choice may take
    int64_t rule_threshold;    // > 0: the slices follow split_rule over the tiles in use
    int32_t* splits_out;       // the slices taken, written by workgroup 0 (or null)
    int64_t split_stride;      // elements between split slices of out / out2
    void* out;                 // plain: fp32 [split][rows][M]; gated: fp32 G partials
                               // [split][rows][M] (used when more than one slice)
    float* out2;               // gated: fp32 U partials [split][rows][M]
    uint16_t* h;               // gated: bf16 H [rows][M] (written here when one slice is taken)
    int kin;                   // gated: reduction groups per workgroup (2, or 1 when 0 or 1)
    int narrow;                // host only: plain kernels keep 4-wave workgroups (more,
                               // smaller work items) instead of 8
};

__device__ __forceinline__ bf16x8 ld16(const uint16_t* p) {
    return *reinterpret_cast<const bf16x8*>(p);
}
// Weight bytes are streamed once per launch.  Read as whole kilobytes (the
// packed layout), non-temporal loads (streaming cache policy) reach a
// measured ~6.3 TB/s against ~5.5 TB/s for plain loads of the same 512 MiB;
// on row-major rows, where one load instruction covers 64 bytes of each of
// 16 rows, they are slower than plain loads (~5.0 against ~5.2-5.4 TB/s),
// so only the packed path uses them.
__device__ __forceinline__ bf16x8 ld16_stream(const uint16_t* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const bf16x8*>(p));
}
// Weight loads of 128-token tiles follow the launch's weight footprint:
// when the experts in use hold at most this many bytes of the launch's
// matrices they are loaded through the caches and stay in the chip's
// last-level cache for the next call (decode steps keep selecting the same
// experts); more than that streams past the caches (non-temporal), which
// keeps them for the token rows.  Smaller tiles always stream: they serve
// calls whose experts' weights far exceed the cache.
#ifndef EAT_CACHE_WEIGHT_BYTES
#define EAT_CACHE_WEIGHT_BYTES (96ll << 20)
#endif
#ifndef EAT_CACHE_MIN_NSUB
#define EAT_CACHE_MIN_NSUB 8
#endif
template <bool STREAM>
__device__ __forceinline__ bf16x8 ld16_w(const uint16_t* p) {
    if constexpr (STREAM) return ld16_stream(p);
    else return ld16(p);
}



// H = bf16(silu(G) * U) for a lane's 4 consecutive features.
__device__ __forceinline__ void store_h(uint16_t* dst, const f32x4& gsum, const f32x4& usum) {
    uint16_t hv[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) hv[q] = f32_to_bf16(silu(gsum[q]) * usum[q]);
    uint2 pk;
    pk.x = static_cast<uint32_t>(hv[0]) | (static_cast<uint32_t>(hv[1]) << 16);
    pk.y = static_cast<uint32_t>(hv[2]) | (static_cast<uint32_t>(hv[3]) << 16);
    *reinterpret_cast<uint2*>(dst) = pk;
}

// One workgroup = WPB waves = 16 WPB consecutive weight rows (16 per wave) of one
// expert, applied to one tile of up to 16*NSUB of that expert's tokens.
// The reduction dimension is walked in chunks of 32*KS:
//   * the tile's token rows for the next chunk are fetched into registers
//     and parked in the other half of a double-buffered LDS slab;
//   * the wave's weight fragments for the next chunk are fetched into a
//     second register set;
// both while the MFMAs of the current chunk run, so every wave keeps
// 16*KS*(GATED ? 2 : 1) bytes per lane of weights in flight.
// Token sub-tiles beyond the tile's row count are skipped (uniform branch),
// so a tile of 1 token costs one MFMA per k-step and matrix.
// Token rows two chunks ahead (see the main loop) in every variant.  Measured
// against one chunk ahead: the 128-token gated tiles +12% on the fine-grained
// layer's 256-token Top-K decode and +4-6% in EAT; the plain projection's
// 128-token tiles +8% (down) on the shared-expert layer's EAT decode, the
// 16-layer stack +1%; the 2-step chunks of 128-token gated tiles spill, and
// with one chunk ahead they gain less (EAT_KS_G8 = 2: +2-5%).
#ifndef EAT_DEEP_NSUB
#define EAT_DEEP_NSUB 8
#endif
#ifndef EAT_DEEP_PLAIN_NSUB
#define EAT_DEEP_PLAIN_NSUB 8
#endif
template <bool GATED, int NSUB>
constexpr bool stream_deep() { return GATED ? NSUB <= EAT_DEEP_NSUB : NSUB <= EAT_DEEP_PLAIN_NSUB; }

// At least 3 waves per SIMD: the register budget then keeps the MFMA
// accumulators in VGPRs (no AGPR copies) and the 64-token gated variant
// holds 3 waves per SIMD instead of 2 (measured: more weight bytes in flight).
// KIN = 2: the workgroup holds two groups of WPB waves over the same weight
// rows, each taking one half of the item's reduction slice (its own token
// staging); group 1 hands its accumulators to group 0 through LDS at the
// end of the item.  This doubles the waves of a launch whose experts are few
// without the fp32 partials and the reduce launch of a split across
// workgroups.
template <bool GATED, int NSUB, int KS, int WPB, bool PACKED, int KIN = 1>
// (Two groups of the 128-token gated tiles need one register more than 3
// waves per SIMD leave, and their 8 waves' LDS keeps one workgroup per CU
// anyway: they take 2.)
__global__ __launch_bounds__(WPB * 64 * KIN)
__attribute__((amdgpu_waves_per_eu((KIN == 2 && NSUB >= 8) ? 2 : 3, 8))) void stream_kernel(StreamArgs a) {
    static_assert(KIN == 1 || (KIN == 2 && GATED), "two reduction groups in the gated kernel only");
    constexpr int NT = WPB * 64;                      // threads per reduction group
    constexpr int BN = 16 * NSUB;
    constexpr int KC = 32 * KS;
    constexpr int LDS_ROW = KC + 8;                   // +16 B per row against bank conflicts
    constexpr int VPR = KC / 8;                       // 16-byte vectors per token row per chunk
    constexpr int RMAX = (BN * VPR + NT - 1) / NT;    // vectors per thread per chunk
    constexpr bool DEEP = stream_deep<GATED, NSUB>();
    // the token slabs (two per reduction group), also holding group 1's sums
    // at the end of an item when KIN = 2
    constexpr int kSlabs = KIN * 2 * BN * LDS_ROW;
    constexpr int kSums = KIN == 2 ? NT * NSUB * 8 * 2 : 0;     // in 16-bit units
    __shared__ __attribute__((aligned(16))) uint16_t xs[kSlabs > kSums ? kSlabs : kSums];
    auto slab = [&](int grp, int buf) __attribute__((always_inline)) {
        return xs + (grp * 2 + buf) * (BN * LDS_ROW);
    };
    __shared__ int tstart[kMaxExperts + 1];
    __shared__ int used_groups;
    const int lane = lane_id();
    // reduction group (uniform over the wave), the wave's place in it and
    // the thread's
    const int kg = KIN == 1 ? 0 : __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / NT);
    const int tid = KIN == 1 ? static_cast<int>(threadIdx.x) : static_cast<int>(threadIdx.x) - kg * NT;
    const int wave = tid / kWave;

    int ntiles, used = 1;
    if (a.offsets) {
        tile_starts<true>(a.offsets, a.groups, BN, tstart, &used_groups);
        ntiles = tstart[a.groups];
        used = used_groups;
    } else {
        ntiles = (a.nrows + BN - 1) / BN;
    }
    // slices of the reduction dimension: fixed, or chosen from the tiles in
    // use (every workgroup computes the same value)
    // (the rule counts both reduction groups' waves)
    const int splits =
        a.rule_threshold > 0 ? split_rule(a.M * KIN, a.K / KIN, ntiles, a.splits, a.rule_threshold, GATED) : a.splits;
    if (a.splits_out && blockIdx.x == 0 && threadIdx.x == 0) *a.splits_out = splits;
    const int ksplit = a.K / splits;

    const int i = lane & 15, g = lane >> 4;
    const int nch = ksplit / KIN / KC;
    const int nrb = a.M / (16 * WPB);                 // weight-row blocks

    // Work items (token tile, reduction slice, row block), row block
    // fastest; the grid holds about as many workgroups as the chip keeps
    // resident, each taking items grid-stride.  Only the tiles in use count,
    // so a call whose tokens land on few experts leaves no idle workgroups
    // behind the working ones.
    // (the launcher keeps the item count below 2^31)
    const unsigned items = static_cast<unsigned>(ntiles) * splits * nrb;
    const int64_t footprint = static_cast<int64_t>(used) * a.M * a.K * (GATED ? 4 : 2);
    const bool stream_w = NSUB < EAT_CACHE_MIN_NSUB || footprint > EAT_CACHE_WEIGHT_BYTES;
    auto run = [&](auto stream_tag) __attribute__((always_inline)) {
        constexpr bool kStreamW = decltype(stream_tag)::value;
        for (unsigned w = blockIdx.x; w < items; w += gridDim.x) {
            const int rb = static_cast<int>(w % nrb);
            const unsigned rest = w / nrb;
            const int split = static_cast<int>(rest % splits);
            const int tile = static_cast<int>(rest / splits);
            const int m0 = rb * (16 * WPB) + wave * 16;
            const int kbeg = split * ksplit + kg * (ksplit / KIN);
            int e = 0, r0, n;
            if (a.offsets) {
                e = tile_group(tstart, a.groups, tile);
                r0 = a.offsets[e] + (tile - tstart[e]) * BN;
                n = min(BN, a.offsets[e + 1] - r0);
            } else {
                r0 = tile * BN;
                n = min(BN, a.nrows - r0);
            }
            const int nsub = (n + 15) >> 4;
            // Row-major weights: this lane's 8 elements of row m0 + i at k-offset
            // 8 g of each 32-wide k-step.  Packed weights: the wave's 16 rows form
            // one 1 KB block per k-step, lane l's fragment at 16 l bytes.
            const size_t wrow = PACKED ? (static_cast<size_t>(e) * (a.M / 16) + m0 / 16) * (a.K / 32) * 512 + 8 * lane
                                       : (static_cast<size_t>(e) * a.M + m0 + i) * a.K + 8 * g;
            const uint16_t* pa = a.wa + wrow;
            const uint16_t* pb = GATED ? a.wb + wrow : nullptr;

            // token-row vectors this thread moves into LDS each chunk
            const uint16_t* xsrc[RMAX];
            int xdst[RMAX];
            bool xon[RMAX];
#pragma unroll
            for (int r = 0; r < RMAX; ++r) {
                const int v = tid + NT * r;
                const int row = v / VPR, col = v % VPR;
                xon[r] = row < n;
                const int srow = xon[r] ? (a.gather ? a.gather[r0 + row] : r0 + row) : 0;
                xsrc[r] = a.src + static_cast<size_t>(srow) * a.K + kbeg + 8 * col;
                xdst[r] = row * LDS_ROW + 8 * col;
            }
            // Every lane loads (rows past the tile read a valid row and are not
            // stored), so xr stays in registers instead of private memory.
            // (native vector type: HIP's uint4 struct would be copied with
            // memcpy and kept in private memory)
            bf16x8 xr[RMAX];
            auto load_xr = [&](int c, bf16x8 (&R)[RMAX]) __attribute__((always_inline)) {
#pragma unroll
                for (int r = 0; r < RMAX; ++r) R[r] = ld16(xsrc[r] + c * KC);
            };
            auto store_xr = [&](int buf, const bf16x8 (&R)[RMAX]) __attribute__((always_inline)) {
#pragma unroll
                for (int r = 0; r < RMAX; ++r)
                    if (xon[r]) *reinterpret_cast<bf16x8*>(slab(kg, buf) + xdst[r]) = R[r];
            };
            auto load_x = [&](int c) __attribute__((always_inline)) { load_xr(c, xr); };
            auto store_x = [&](int buf) __attribute__((always_inline)) { store_xr(buf, xr); };
            auto load_w = [&](int c, bf16x8 (&A)[KS], bf16x8 (&B)[KS]) __attribute__((always_inline)) {
                const int k = kbeg + c * KC;
#pragma unroll
                for (int j = 0; j < KS; ++j) {
                    if constexpr (PACKED) {
                        const size_t o = static_cast<size_t>(k / 32 + j) * 512;
                        A[j] = ld16_w<kStreamW>(pa + o);
                        if constexpr (GATED) B[j] = ld16_w<kStreamW>(pb + o);
                    } else {
                        A[j] = ld16(pa + k + 32 * j);
                        if constexpr (GATED) B[j] = ld16(pb + k + 32 * j);
                    }
                }
            };

            f32x4 acc_a[NSUB], acc_b[NSUB];
#pragma unroll
            for (int s = 0; s < NSUB; ++s) {
                acc_a[s] = f32x4{0.f, 0.f, 0.f, 0.f};
                acc_b[s] = f32x4{0.f, 0.f, 0.f, 0.f};
            }
            // Gated tiles read every populated sub-tile's token fragment before
            // the first MFMA of a k-step and pin the reads there (an empty asm
            // that takes them as inputs), so the LDS latency is paid once per
            // k-step.  Left to itself the compiler sinks each read into its
            // sub-tile's guard, behind the previous sub-tile's MFMAs: one full
            // LDS round trip per sub-tile.  Rows of the last sub-tile past its
            // tokens hold stale values that only reach output columns that are
            // never stored.  The plain projection keeps the guarded reads: with
            // one MFMA per read the pins cost it more than the latency they hide
            // (measured).
            auto compute = [&](int buf, const bf16x8 (&A)[KS], const bf16x8 (&B)[KS]) __attribute__((always_inline)) {
                const uint16_t* xb = slab(kg, buf);
#pragma unroll
                for (int j = 0; j < KS; ++j) {
                    if constexpr (GATED) {
                        bf16x8 X[NSUB];
#pragma unroll
                        for (int s = 0; s < NSUB; ++s)
                            X[s] = s < nsub ? *reinterpret_cast<const bf16x8*>(xb + (s * 16 + i) * LDS_ROW + 32 * j + 8 * g)
                                            : bf16x8{};
#pragma unroll
                        for (int s = 0; s < NSUB; ++s) asm volatile("" ::"v"(X[s]));
#pragma unroll
                        for (int s = 0; s < NSUB; ++s) {
                            if (s < nsub) {
                                acc_a[s] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[j], X[s], acc_a[s], 0, 0, 0);
                                acc_b[s] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(B[j], X[s], acc_b[s], 0, 0, 0);
                            }
                        }
                    } else {
#pragma unroll
                        for (int s = 0; s < NSUB; ++s) {
                            if (s < nsub) {
                                const bf16x8 X =
                                    *reinterpret_cast<const bf16x8*>(xb + (s * 16 + i) * LDS_ROW + 32 * j + 8 * g);
                                acc_a[s] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[j], X, acc_a[s], 0, 0, 0);
                            }
                        }
                    }
                }
            };

            if constexpr (DEEP) {
                // Token rows two chunks ahead: chunk c + 2's rows are loaded into
                // one of two register sets while chunk c + 1's (loaded a chunk
                // earlier) go to LDS, so no chunk waits on a token-row load it
                // issued itself; weights one chunk ahead in two register sets.
                // Every load is issued unconditionally (a conditional load leaves
                // a merge the register allocator resolves with copies, and a copy
                // waits for its load): past the last chunk the weight loads read
                // a token row instead and the token loads read the last chunk
                // again (valid, L2-resident, unused).
                auto load_w_at = [&](int c, bf16x8 (&A)[KS], bf16x8 (&B)[KS]) __attribute__((always_inline)) {
                    const bool in = c < nch;
                    const int k = kbeg + (in ? c : 0) * KC;
#pragma unroll
                    for (int j = 0; j < KS; ++j) {
                        const size_t o = PACKED ? static_cast<size_t>(k / 32 + j) * 512 : static_cast<size_t>(k + 32 * j);
                        const uint16_t* qa = in ? pa + o : xsrc[0];
                        A[j] = PACKED ? ld16_w<kStreamW>(qa) : ld16(qa);
                        if constexpr (GATED) {
                            const uint16_t* qb = in ? pb + o : xsrc[0];
                            B[j] = PACKED ? ld16_w<kStreamW>(qb) : ld16(qb);
                        }
                    }
                };
                bf16x8 A0[KS], B0[KS], A1[KS], B1[KS], X0[RMAX], X1[RMAX];
                load_xr(0, X0);
                load_w_at(0, A0, B0);
                load_xr(min(1, nch - 1), X1);
                store_xr(0, X0);
                lds_barrier();
                // chunk c: weights in set c % 2, token rows in LDS buffer c % 2;
                // issue token rows c + 2 into set c % 2 and weights c + 1 into set
                // (c + 1) % 2, then move token set (c + 1) % 2 to LDS (c + 1) % 2
                auto stage = [&](int c, const bf16x8 (&Ac)[KS], const bf16x8 (&Bc)[KS], bf16x8 (&An)[KS],
                                 bf16x8 (&Bn)[KS], bf16x8 (&Xn2)[RMAX], const bf16x8 (&Xn1)[RMAX],
                                 int cur) __attribute__((always_inline)) {
                    load_xr(min(c + 2, nch - 1), Xn2);
                    load_w_at(c + 1, An, Bn);
                    compute(cur, Ac, Bc);
                    if (c + 1 < nch) store_xr(cur ^ 1, Xn1);
                    lds_barrier();
                };
                for (int c = 0; c < nch; c += 2) {
                    stage(c, A0, B0, A1, B1, X0, X1, 0);
                    if (c + 1 >= nch) break;
                    stage(c + 1, A1, B1, A0, B0, X1, X0, 1);
                }
            } else {
            // Two register sets in ping-pong: while the MFMAs consume one chunk's
            // weights, the next chunk's are in flight in the other set (no
            // register copies, so the loads are not waited for early).
            bf16x8 A0[KS], B0[KS], A1[KS], B1[KS];
            load_x(0);
            load_w(0, A0, B0);
            store_x(0);
            lds_barrier();
            for (int c = 0; c < nch; c += 2) {
                const bool has1 = c + 1 < nch;
                if (has1) {
                    load_x(c + 1);
                    load_w(c + 1, A1, B1);
                }
                compute(0, A0, B0);
                if (has1) store_x(1);
                lds_barrier();
                if (!has1) break;
                const bool has2 = c + 2 < nch;
                if (has2) {
                    load_x(c + 2);
                    load_w(c + 2, A0, B0);
                }
                compute(1, A1, B1);
                if (has2) store_x(0);
                lds_barrier();
            }
            }

            if constexpr (KIN == 2) {
                // group 1's sums to group 0 through the token slabs (every
                // wave is past its last LDS read: the loop ends with a
                // barrier), added after group 0's own; the second barrier
                // keeps the next item's token staging off the slabs until
                // they have been read
                float* const cmb = reinterpret_cast<float*>(xs);
                const int base = (wave * kWave + lane) * NSUB * 8;
                if (kg == 1) {
#pragma unroll
                    for (int s = 0; s < NSUB; ++s) {
                        *reinterpret_cast<f32x4*>(cmb + base + 8 * s) = acc_a[s];
                        *reinterpret_cast<f32x4*>(cmb + base + 8 * s + 4) = acc_b[s];
                    }
                }
                lds_barrier();
                if (kg == 0) {
#pragma unroll
                    for (int s = 0; s < NSUB; ++s) {
                        acc_a[s] += *reinterpret_cast<const f32x4*>(cmb + base + 8 * s);
                        acc_b[s] += *reinterpret_cast<const f32x4*>(cmb + base + 8 * s + 4);
                    }
                }
                lds_barrier();
                if (kg == 1) continue;               // group 0 stores the item
            }
            // result: lane holds weight rows m0 + 4g + q (q < 4) for token column s*16 + i
            if constexpr (GATED) {
                if (splits == 1) {
#pragma unroll
                    for (int s = 0; s < NSUB; ++s) {
                        const int c = s * 16 + i;
                        if (c >= n) continue;
                        store_h(a.h + static_cast<size_t>(r0 + c) * a.M + m0 + 4 * g, acc_a[s], acc_b[s]);
                    }
                } else {
                    // this slice's G/U partial sums (swiglu_reduce_kernel adds
                    // the slices in order and forms H)
#pragma unroll
                    for (int s = 0; s < NSUB; ++s) {
                        const int c = s * 16 + i;
                        if (c >= n) continue;
                        const size_t po = split * a.split_stride + static_cast<size_t>(r0 + c) * a.M + m0 + 4 * g;
                        *reinterpret_cast<float4*>(static_cast<float*>(a.out) + po) =
                            make_float4(acc_a[s][0], acc_a[s][1], acc_a[s][2], acc_a[s][3]);
                        *reinterpret_cast<float4*>(a.out2 + po) =
                            make_float4(acc_b[s][0], acc_b[s][1], acc_b[s][2], acc_b[s][3]);
                    }
                }
            } else {
#pragma unroll
                for (int s = 0; s < NSUB; ++s) {
                    const int c = s * 16 + i;
                    if (c >= n) continue;
                    float* op = static_cast<float*>(a.out) + split * a.split_stride +
                                static_cast<size_t>(r0 + c) * a.M + m0 + 4 * g;
                    *reinterpret_cast<float4*>(op) = make_float4(acc_a[s][0], acc_a[s][1], acc_a[s][2], acc_a[s][3]);
                }
            }
        }
    };
    if constexpr (NSUB >= EAT_CACHE_MIN_NSUB) {
        if (stream_w) run(std::true_type{});
        else run(std::false_type{});
    } else {
        run(std::true_type{});
    }
}

// out[i] = sum_s part[s][i] (float4 elements, slices added in slice order).
__global__ __launch_bounds__(256) void sum_slices_kernel(const float* __restrict__ part, int splits, int64_t stride,
                                                         int64_t n4, float* __restrict__ out) {
    for (int64_t v = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; v < n4; v += int64_t(gridDim.x) * blockDim.x) {
        float4 o = *reinterpret_cast<const float4*>(part + 4 * v);
        for (int sp = 1; sp < splits; ++sp) {
            const float4 q = *reinterpret_cast<const float4*>(part + sp * stride + 4 * v);
            o.x += q.x; o.y += q.y; o.z += q.z; o.w += q.w;
        }
        *reinterpret_cast<float4*>(out + 4 * v) = o;
    }
}

// H[r][f] = bf16(silu(sum_s G[s][r][f]) * sum_s U[s][r][f]) over the rows
// in use (*rows_dev of them, or rows_host when rows_dev is null), slices
// added in slice order.  The slice count is *splits_dev (the gated launch's
// own choice) when set, else splits_host; with one slice the projection
// wrote H itself and there is nothing to do.
__global__ __launch_bounds__(256) void swiglu_reduce_kernel(const float* __restrict__ gp,
                                                            const float* __restrict__ up,
                                                            const int32_t* __restrict__ rows_dev, int rows_host,
                                                            int M, const int32_t* __restrict__ splits_dev,
                                                            int splits_host, int64_t split_stride,
                                                            uint16_t* __restrict__ h) {
    const int splits = splits_dev ? *splits_dev : splits_host;
    if (splits <= 1) return;                          // uniform: one load, then every thread leaves
    const int64_t total = static_cast<int64_t>(rows_dev ? *rows_dev : rows_host) * (M / 4);
    for (int64_t v = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; v < total;
         v += int64_t(gridDim.x) * blockDim.x) {
        const int64_t o = 4 * v;
        float4 gs = *reinterpret_cast<const float4*>(gp + o);
        float4 us = *reinterpret_cast<const float4*>(up + o);
        for (int sp = 1; sp < splits; ++sp) {
            const float4 ga = *reinterpret_cast<const float4*>(gp + sp * split_stride + o);
            const float4 ua = *reinterpret_cast<const float4*>(up + sp * split_stride + o);
            gs.x += ga.x; gs.y += ga.y; gs.z += ga.z; gs.w += ga.w;
            us.x += ua.x; us.y += ua.y; us.z += ua.z; us.w += ua.w;
        }
        store_h(h + o, f32x4{gs.x, gs.y, gs.z, gs.w}, f32x4{us.x, us.y, us.z, us.w});
    }
}

// Largest chunk (in 32-wide k-steps) that divides the reduction slice.
static int pick_ks(int ksplit) {
    for (int ks : {8, 4, 2, 1})
        if (ksplit % (32 * ks) == 0) return ks;
    return 1;
}

// Chunk depth (k-steps of 32) per variant.  Each wave keeps one chunk of
// weight fragments in flight, so the bytes in flight per CU are about
// waves/SIMD x 4 x KS x 1 KB (x2 when gated); the table maximises that
// product for the register and LDS footprint of each variant, spill-free.
// The gated 64-token variant keeps a second token-row register set (two
// chunks ahead) and is faster with 2 k-steps at 4 waves per SIMD than with
// 4 at 3 (measured on the Mixtral-shaped decode layer).
#ifndef EAT_KS_G1
#define EAT_KS_G1 4
#endif
#ifndef EAT_KS_G2
#define EAT_KS_G2 4
#endif
#ifndef EAT_KS_G8
#define EAT_KS_G8 1
#endif
#ifndef EAT_KS_G4
#define EAT_KS_G4 2
#endif
#ifndef EAT_KS_P1
#define EAT_KS_P1 8
#endif
#ifndef EAT_KS_P2
#define EAT_KS_P2 8
#endif
#ifndef EAT_KS_P4
#define EAT_KS_P4 4
#endif
template <bool GATED, int NSUB>
constexpr int max_ks() {
    if (GATED) return NSUB >= 8 ? EAT_KS_G8 : NSUB >= 4 ? EAT_KS_G4 : NSUB >= 2 ? EAT_KS_G2 : EAT_KS_G1;
    return NSUB >= 8 ? 2 : NSUB >= 4 ? EAT_KS_P4 : NSUB >= 2 ? EAT_KS_P2 : EAT_KS_P1;
}

// Waves per workgroup: the down projection with 64+-token tiles shares one
// token slab between 8 waves (half the slab traffic per weight byte).  The
// gated kernel with up to 64-token tiles runs 2 waves (32 weight rows) per
// workgroup: twice the work items of 4 waves, so the last ones spread more
// evenly over the CUs (Mixtral-shaped decode +1%, its Top-K +4%, the 16-layer
// stack's Top-K +6%).  8 waves for the gated 128-token tiles (EAT_WPB_G8):
// Top-K on the fine-grained 256-token decode +7%, EAT -7% and the
// shared-expert layer -2 to -5% (EAT's few experts want more, smaller
// workgroups); they keep 4.
#ifndef EAT_WPB_G8
#define EAT_WPB_G8 4
#endif
template <bool GATED, int NSUB>
constexpr int stream_wpb() { return (!GATED && NSUB >= 4) ? 8 : (GATED && NSUB >= 8) ? EAT_WPB_G8 : GATED ? 2 : 4; }

// Workgroups of one stream-kernel instance the whole chip keeps resident
// (occupancy per CU x CUs), asked once per instance on the device current
// at the first call (every device a process uses is assumed to be the same
// part; a smaller grid on a larger part is still correct, only less full).
template <bool GATED, int NSUB, int KS, int WPB, bool PACKED, int KIN>
int64_t stream_resident() {
    static const int64_t v = [] {
        int dev = 0, cus = 0, per_cu = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
            cus = 256;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, stream_kernel<GATED, NSUB, KS, WPB, PACKED, KIN>,
                                                         WPB * 64 * KIN, 0) != hipSuccess ||
            per_cu < 1)
            per_cu = 1;
        return static_cast<int64_t>(cus) * per_cu;
    }();
    return v;
}

// Compute units of the device current at the first call.
static int chip_cus() {
    static const int v = [] {
        int dev = 0, cus = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
            cus = 256;
        return cus;
    }();
    return v;
}

// Grid: as many workgroups as there can be work items (max_tiles token
// tiles x slices x row blocks), at most what the chip keeps resident.
template <bool GATED, int NSUB, int KS, int WPB, bool PACKED, int KIN>
hipError_t launch_stream_wk(const StreamArgs& a, int64_t max_tiles, hipStream_t s) {
    const int64_t items = max_tiles * a.splits * (a.M / (16 * WPB));
    if (items >= (int64_t{1} << 31)) return hipErrorInvalidValue;
    int64_t blocks = std::max<int64_t>(1, std::min(items, stream_resident<GATED, NSUB, KS, WPB, PACKED, KIN>()));
    stream_kernel<GATED, NSUB, KS, WPB, PACKED, KIN>
        <<<dim3(static_cast<unsigned>(blocks)), dim3(WPB * 64 * KIN), 0, s>>>(a);
    return hipGetLastError();
}

template <bool GATED, int NSUB, int KS, int WPB, bool PACKED>
hipError_t launch_stream_w(const StreamArgs& a, int64_t max_tiles, hipStream_t s) {
    if constexpr (GATED) {
        if (a.kin == 2) return launch_stream_wk<GATED, NSUB, KS, WPB, PACKED, 2>(a, max_tiles, s);
    }
    return launch_stream_wk<GATED, NSUB, KS, WPB, PACKED, 1>(a, max_tiles, s);
}

template <bool GATED, int NSUB, int KS, bool PACKED>
hipError_t launch_stream_k(const StreamArgs& a, int64_t max_tiles, hipStream_t s) {
    if constexpr (KS > max_ks<GATED, NSUB>()) {
        return hipErrorInvalidValue;
    } else if constexpr (stream_wpb<GATED, NSUB>() == 8) {
        if (a.M % 128 == 0 && !a.narrow) return launch_stream_w<GATED, NSUB, KS, 8, PACKED>(a, max_tiles, s);
        return launch_stream_w<GATED, NSUB, KS, 4, PACKED>(a, max_tiles, s);
    } else if constexpr (stream_wpb<GATED, NSUB>() == 2) {
        if (a.M % 32 == 0) return launch_stream_w<GATED, NSUB, KS, 2, PACKED>(a, max_tiles, s);
        return launch_stream_w<GATED, NSUB, KS, 4, PACKED>(a, max_tiles, s);
    } else {
        return launch_stream_w<GATED, NSUB, KS, 4, PACKED>(a, max_tiles, s);
    }
}

template <bool GATED, int NSUB, bool PACKED>
hipError_t launch_stream_n(const StreamArgs& a, int64_t max_tiles, hipStream_t s) {
    // the device may take fewer slices than a.splits; K / a.splits divides
    // every longer slice, so its chunk depth fits them all
    const int ks = std::min(pick_ks(a.K / a.splits / (a.kin == 2 ? 2 : 1)), max_ks<GATED, NSUB>());
    switch (ks) {
        case 8: return launch_stream_k<GATED, NSUB, 8, PACKED>(a, max_tiles, s);
        case 4: return launch_stream_k<GATED, NSUB, 4, PACKED>(a, max_tiles, s);
        case 2: return launch_stream_k<GATED, NSUB, 2, PACKED>(a, max_tiles, s);
        default: return launch_stream_k<GATED, NSUB, 1, PACKED>(a, max_tiles, s);
    }
}

template <bool GATED, bool PACKED>
hipError_t launch_stream_p(const StreamArgs& a, int nsub, int64_t max_tiles, hipStream_t s) {
    switch (nsub) {
        case 1: return launch_stream_n<GATED, 1, PACKED>(a, max_tiles, s);
        case 2: return launch_stream_n<GATED, 2, PACKED>(a, max_tiles, s);
        case 4: return launch_stream_n<GATED, 4, PACKED>(a, max_tiles, s);
        default: return launch_stream_n<GATED, 8, PACKED>(a, max_tiles, s);
    }
}

// Up to `a.splits` slices; max_tiles bounds the token tiles a
// call can hold (their count is only known on the device); `packed` selects
// the packed weight layout (pack.hip).
template <bool GATED>
hipError_t launch_stream(const StreamArgs& a, int nsub, int64_t max_tiles, bool packed, hipStream_t s) {
    return packed ? launch_stream_p<GATED, true>(a, nsub, max_tiles, s)
                  : launch_stream_p<GATED, false>(a, nsub, max_tiles, s);
}

}  // namespace

// Token sub-tiles per stream tile: one tile holds every token an expert
// can receive in a call of T tokens (at most T), up to 128; beyond that an
// expert's tokens take several tiles.
static int pick_nsub(int64_t T) {
    if (T <= 16) return 1;
    if (T <= 32) return 2;
    if (T <= 64) return 4;
    return 8;
}

// Most slices a launch of T tokens may take: the rule over the fewest tiles
// the call can hold (the rule only shrinks as tiles grow).  Every token of
// a Top-K call selects exactly K experts, so it holds at least
// max(K, ceil(T K / bn)) tiles; an EAT or Top-P token selects at least one
// expert, so at least ceil(T / bn).  The device takes the rule over the
// tiles actually in use (stream_kernel).
static int min_tiles(const eat_params_t& p, int32_t T) {
    const int64_t bn = 16 * pick_nsub(T);
    const int64_t t = std::max<int64_t>(1, T);
    return static_cast<int>(p.mode == EAT_MODE_TOPK ? std::max<int64_t>(p.top_k, (t * p.top_k + bn - 1) / bn)
                                                    : (t + bn - 1) / bn);
}

// Tiles a call is expected to hold: EAT concentrates its picks on about K
// experts; Top-K and Top-P tokens spread over min(E, T K).  The up/gate
// projection plans its slices for this many (the device may take fewer,
// never more): its slices need a reduce kernel, and planning for a
// one-expert union would launch it for nothing in most calls.
static int expected_tiles(const eat_params_t& p, int32_t T) {
    const int64_t assign = std::max<int64_t>(1, static_cast<int64_t>(T) * p.top_k);
    const int64_t active = std::min<int64_t>(
        {static_cast<int64_t>(p.E), assign, p.mode == EAT_MODE_EAT ? static_cast<int64_t>(p.top_k) : assign});
    const int64_t bn = 16 * pick_nsub(T);
    return static_cast<int>(std::max<int64_t>(active, (assign + bn - 1) / bn));
}

// Calls averaging at least this many rows per expert take the wide MFMA
// tiles.  Measured at 32 (the fine-grained layer's 256-token decode then
// goes wide): Top-K +4%, EAT -2% -- EAT's ~8 experts leave the wide tiles
// ~66 work items for 256 CUs, and its down projection slows from 31 to 42 us.
#ifndef EAT_WIDE_ROWS
#define EAT_WIDE_ROWS 256
#endif
// Prefill-sized calls (EAT_WIDE_ROWS or more rows per expert on average;
// the always-on expert from 384 tokens) go through the wide MFMA tiles.
static bool use_wide(const eat_params_t& p, int32_t T) {
    return p.expert_dtype == EAT_BF16 && static_cast<int64_t>(T) * p.top_k >= int64_t{EAT_WIDE_ROWS} * p.E &&
           wide_fits(true, p.d_ffn, p.d_model) && wide_fits(false, p.d_model, p.d_ffn);
}
static bool shared_wide(const eat_params_t& p, int32_t T) {
    return T >= 384 && p.d_shared > 0 && wide_fits(true, p.d_shared, p.d_model) &&
           wide_fits(false, p.d_model, p.d_shared);
}

bool rows_bf16(const eat_params_t& p, int32_t T) { return use_wide(p, T); }

int norm_parts(const eat_params_t& p, int32_t T) {
    return rows_bf16(p, T) ? p.d_model / 32 : combine_chunks(p);
}

int down_splits(const eat_params_t& p, int32_t T) {
    if (p.expert_dtype != EAT_BF16 || use_wide(p, T)) return 1;
    return split_rule(p.d_model, p.d_ffn, min_tiles(p, T), 8, EAT_SPLIT_WAVES, false);
}

// Reduction groups per workgroup of the gated stream kernel: two where the
// rule would split the reduction across workgroups (few experts, few waves),
// which halves the slices the projection writes and a reduce adds (none left
// at one slice); one otherwise.
#ifndef EAT_UP_KIN
#define EAT_UP_KIN 1
#endif
static int up_groups(int M, int K, int64_t tiles, int64_t threshold) {
    if (!EAT_UP_KIN || (K / 2) % 64 != 0) return 1;
    return split_rule(M, K, tiles, EAT_UP_SPLIT_MAX, threshold, true) >= 2 ? 2 : 1;
}

static int64_t up_threshold(int32_t T) { return pick_nsub(T) >= 8 ? EAT_UP_SPLIT_WAVES_T128 : EAT_UP_SPLIT_WAVES; }

static int up_kin(const eat_params_t& p, int32_t T) {
    if (p.expert_dtype != EAT_BF16 || use_wide(p, T)) return 1;
    return up_groups(p.d_ffn, p.d_model, expected_tiles(p, T), up_threshold(T));
}

int up_splits(const eat_params_t& p, int32_t T) {
    if (p.expert_dtype != EAT_BF16 || use_wide(p, T)) return 1;
    const int kin = up_kin(p, T);
    return split_rule(p.d_ffn * kin, p.d_model / kin, expected_tiles(p, T), EAT_UP_SPLIT_MAX, up_threshold(T), true);
}

// Dense projection (one group of T identity rows): the wide tiles from 384
// rows, else the plain stream kernel with its reduction dimension split
// until ~4096 wave tiles exist.
static bool dense_wide(int M, int K, int32_t T) { return T >= 384 && wide_fits(false, M, K); }

int dense_splits(int M, int K, int32_t T) {
    if (dense_wide(M, K, T)) return 1;
    const int64_t bn = 16 * pick_nsub(T);
    const int64_t waves = static_cast<int64_t>(M / 16) * ((T + bn - 1) / bn);
    int s = 1;
    while (s < 8 && K % (64 * 2 * s) == 0 && waves * s < EAT_SPLIT_WAVES) s *= 2;
    return s;
}

hipError_t launch_dense_bf16(const uint16_t* src, int32_t T, const uint16_t* w, int M, int K, float* out,
                             int splits, int64_t split_stride, hipStream_t s) {
    if (dense_wide(M, K, T))
        return launch_wide(false, w, nullptr, src, nullptr, nullptr, 1, T, M, K, out, T, false, nullptr, s);
    const int nsub = pick_nsub(T);
    const int bn = 16 * nsub;
    const int tiles = (T + bn - 1) / bn;
    StreamArgs a{};
    a.wa = w; a.src = src; a.nrows = T; a.groups = 1; a.M = M; a.K = K; a.splits = splits;
    a.split_stride = split_stride; a.out = out;
    // 8-wave items that would not reach every CU (the 2048-wide mixing GEMM
    // of a 64-token decode: 128 items) take 4-wave ones instead
    a.narrow = static_cast<int64_t>(tiles) * splits * (M / 128) < chip_cus();
    return launch_stream<false>(a, nsub, tiles, false, s);
}

hipError_t launch_experts_f32(const eat_params_t& p, int32_t T, int64_t rows_cap, const float* x,
                              const float* w1, const float* w3, const float* w2,
                              const int32_t* offsets, const int32_t* tok_idx,
                              const int32_t* row_expert, float* h, float* yp, hipStream_t s,
                              const std::function<void()>& between) {
    F32Args a{x, w1, w3, w2, tok_idx, row_expert, offsets + p.E, 0, p.d_model, p.d_ffn, h, yp};
    (void)T;
    return launch_f32_pair(a, rows_cap, s, between);
}

hipError_t launch_shared_f32(const eat_params_t& p, int32_t T, const float* x, const float* ws1,
                             const float* ws3, const float* ws2, float* hs, float* ys,
                             hipStream_t s) {
    F32Args a{x, ws1, ws3, ws2, nullptr, nullptr, nullptr, T, p.d_model, p.d_shared, hs, ys};
    return launch_f32_pair(a, T, s, nullptr);
}

hipError_t launch_experts_bf16(const eat_params_t& p, int32_t T, int64_t rows_cap, const uint16_t* x,
                               const uint16_t* w1, const uint16_t* w3, const uint16_t* w2,
                               const int32_t* offsets, const int32_t* tok_idx, uint16_t* h,
                               float* gu, float* yp, float* nrm2, int32_t* up_splits_dev, int32_t* down_splits_dev,
                               hipStream_t s, const std::function<void()>& between) {
    const int nsub = pick_nsub(T);
    const int bn = 16 * nsub;
    // no expert holds more than T rows, so it needs at most ceil(T / bn) tiles
    const int64_t per_expert = (T + bn - 1) / bn;
    const int64_t max_tiles = std::min<int64_t>({rows_cap, per_expert * p.E, (rows_cap + bn - 1) / bn + p.E});

    const bool packed = p.weight_layout == EAT_LAYOUT_PACKED;
    if (use_wide(p, T)) {
        hipError_t err = launch_wide(true, w1, w3, x, tok_idx, offsets, p.E, 0, p.d_ffn, p.d_model, h, rows_cap,
                                     packed, nullptr, s);
        if (err != hipSuccess) return err;
        if (between) between();
        return launch_wide(false, w2, nullptr, h, nullptr, offsets, p.E, 0, p.d_model, p.d_ffn, yp, rows_cap, packed,
                           rows_bf16(p, T) ? nrm2 : nullptr, s);
    }
    // both projections take their slices on the device, from the tiles in use
    const int usplits = up_splits(p, T);
    StreamArgs up{};
    up.kin = up_kin(p, T);
    up.wa = w1; up.wb = w3; up.src = x; up.gather = tok_idx; up.offsets = offsets;
    up.groups = p.E; up.M = p.d_ffn; up.K = p.d_model; up.splits = usplits;
    up.rule_threshold = usplits > 1 ? up_threshold(T) : 0;
    up.split_stride = rows_cap * p.d_ffn;
    up.out = gu;
    up.out2 = gu + usplits * up.split_stride;
    up.h = h;
    up.splits_out = up_splits_dev;
    hipError_t err = launch_stream<true>(up, nsub, max_tiles, packed, s);
    if (err != hipSuccess) return err;
    if (usplits > 1) {
        const int64_t vec = rows_cap * (p.d_ffn / 4);
        const int grid = static_cast<int>(std::min<int64_t>((vec + 255) / 256, 4096));
        swiglu_reduce_kernel<<<grid, 256, 0, s>>>(gu, up.out2, offsets + p.E, 0, p.d_ffn, up_splits_dev, usplits,
                                                  up.split_stride, h);
        err = hipGetLastError();
        if (err != hipSuccess) return err;
    }
    if (between) between();

    const int splits = down_splits(p, T);
    StreamArgs dn{};
    dn.wa = w2; dn.wb = nullptr; dn.src = h; dn.gather = nullptr; dn.offsets = offsets;
    dn.groups = p.E; dn.M = p.d_model; dn.K = p.d_ffn; dn.splits = splits;
    dn.rule_threshold = splits > 1 ? EAT_SPLIT_WAVES : 0;
    dn.splits_out = down_splits_dev;
    dn.split_stride = rows_cap * p.d_model; dn.out = yp;
    return launch_stream<false>(dn, nsub, max_tiles, packed, s);
}

// The always-on expert below the wide-tile size: one tile row block per 64
// weight rows is too few workgroups for the chip (88 for a 5632-wide expert,
// 16 for its 2048-row down projection), so both projections split their
// reduction dimension like a routed call whose tokens all go to one expert.
static int shared_up_kin(const eat_params_t& p, int32_t T) {
    if (p.expert_dtype != EAT_BF16 || p.d_shared == 0 || shared_wide(p, T)) return 1;
    eat_params_t one = p;
    one.E = 1;
    one.top_k = 1;
    return up_groups(p.d_shared, p.d_model, expected_tiles(one, T), up_threshold(T));
}

int shared_up_splits(const eat_params_t& p, int32_t T) {
    if (p.expert_dtype != EAT_BF16 || p.d_shared == 0 || shared_wide(p, T)) return 1;
    eat_params_t one = p;
    one.E = 1;
    one.top_k = 1;
    const int kin = shared_up_kin(p, T);
    return split_rule(p.d_shared * kin, p.d_model / kin, expected_tiles(one, T), EAT_UP_SPLIT_MAX,
                      up_threshold(T), true);
}

int shared_splits(const eat_params_t& p, int32_t T) {
    if (p.expert_dtype != EAT_BF16 || p.d_shared == 0 || shared_wide(p, T)) return 1;
    return dense_splits(p.d_model, p.d_shared, T);
}

hipError_t launch_shared_bf16(const eat_params_t& p, int32_t T, const uint16_t* x, const uint16_t* ws1,
                              const uint16_t* ws3, const uint16_t* ws2, uint16_t* hs, float* ys, float* gus,
                              float* ysp, hipStream_t s) {
    const bool packed = p.weight_layout == EAT_LAYOUT_PACKED;
    if (shared_wide(p, T)) {
        hipError_t err =
            launch_wide(true, ws1, ws3, x, nullptr, nullptr, 1, T, p.d_shared, p.d_model, hs, T, packed, nullptr, s);
        if (err != hipSuccess) return err;
        return launch_wide(false, ws2, nullptr, hs, nullptr, nullptr, 1, T, p.d_model, p.d_shared, ys, T, packed,
                           nullptr, s);
    }
    const int nsub = pick_nsub(T);
    const int bn = 16 * nsub;
    const int tiles = (T + bn - 1) / bn;
    const int usplits = shared_up_splits(p, T);
    StreamArgs up{};
    up.kin = shared_up_kin(p, T);
    up.wa = ws1; up.wb = ws3; up.src = x; up.gather = nullptr; up.offsets = nullptr; up.nrows = T;
    up.groups = 1; up.M = p.d_shared; up.K = p.d_model; up.splits = usplits;
    up.split_stride = static_cast<int64_t>(T) * p.d_shared;
    up.out = gus;
    up.out2 = gus + usplits * up.split_stride;
    up.h = hs;
    hipError_t err = launch_stream<true>(up, nsub, tiles, packed, s);
    if (err != hipSuccess) return err;
    if (usplits > 1) {
        const int64_t vec = static_cast<int64_t>(T) * (p.d_shared / 4);
        const int grid = static_cast<int>(std::min<int64_t>((vec + 255) / 256, 4096));
        swiglu_reduce_kernel<<<grid, 256, 0, s>>>(gus, up.out2, nullptr, T, p.d_shared, nullptr, usplits,
                                                  up.split_stride, hs);
        err = hipGetLastError();
        if (err != hipSuccess) return err;
    }
    const int splits = shared_splits(p, T);
    StreamArgs dn{};
    dn.wa = ws2; dn.wb = nullptr; dn.src = hs; dn.gather = nullptr; dn.offsets = nullptr; dn.nrows = T;
    dn.groups = 1; dn.M = p.d_model; dn.K = p.d_shared; dn.splits = splits;
    dn.split_stride = static_cast<int64_t>(T) * p.d_model;
    dn.out = splits > 1 ? ysp : ys;
    err = launch_stream<false>(dn, nsub, tiles, packed, s);
    if (err != hipSuccess || splits == 1) return err;
    const int64_t n4 = dn.split_stride / 4;
    const int grid = static_cast<int>(std::min<int64_t>((n4 + 255) / 256, 2048));
    sum_slices_kernel<<<grid, 256, 0, s>>>(ysp, splits, dn.split_stride, n4, ys);
    return hipGetLastError();
}

}  // namespace eat
