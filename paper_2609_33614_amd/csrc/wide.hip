// Wide MFMA tiles for prefill-sized grouped GEMMs (gfx950).
//
// At prefill sizes (hundreds of rows per expert) the expert projections are
// dense contractions whose speed is set by how fast each CU can pull operand
// bytes from L2 into LDS.  Measured on this part, that rate grows with the
// number of waves issuing loads (about 20 B/clk per CU with 4 waves, 46 with
// 8, 80 with 16), not with the loads each wave keeps in flight; and lines
// that miss L2 come at roughly HBM speed whatever their pattern.  So a
// workgroup here is 16 waves (4 per SIMD) that own a 256-token x 256-row tile
// (the gated projection: 128 rows of W1 and the matching 128 of W3) -- half
// the bytes per flop of a 128 x 128 tile -- all of them loading the stages
// of a double-buffered LDS ring (64-wide reduction chunks, 128-byte rows,
// direct global->LDS loads) and each computing 64 tokens x 64 weight rows
// with v_mfma_f32_32x32x16_bf16 (weights as A, tokens as B: a lane ends with
// 4 consecutive output features of one token).  Four waves per SIMD hide
// each other's LDS and barrier latency without hand scheduling.  The waves
// of a SIMD cover the four token quarters of the tile, so when a tile holds
// fewer rows of its expert, the waves of the empty quarters skip their
// MFMAs and every SIMD's work shrinks with the tile.
//
// The grid is persistent: the work list (per expert, its weight tiles in
// turn and each one's token tiles adjacent) is cut into contiguous parts,
// one per XCD (workgroups are dealt to XCDs round-robin), so the workgroups
// that share an expert's weight tiles share one L2 and read them together.
// A workgroup's ring runs on from one item to the next, so the refill after
// an item overlaps its output stores.  What is left is set by the weight
// lines a CU fetches for the first time: a weight tile serves only the few
// token tiles of its expert, so each chunk brings 32 KB of L2 misses.
#include "eat_device.h"
#include "eat_internal.h"

namespace eat {
namespace {

constexpr int kWM = 256;                  // token rows per tile
constexpr int kWN = 256;                  // weight rows per tile
// Reduction chunk per stage: 64 (128-byte rows, a 2-stage ring) measured a
// few percent faster than 32 (64-byte rows, a 4-stage ring loading three
// chunks ahead) on the three prefill layers, so load latency is not what
// bounds these tiles.
#ifndef EAT_WIDE_BK
#define EAT_WIDE_BK 64
#endif
constexpr int kWK = EAT_WIDE_BK;          // reduction chunk per stage (bf16 elements)
constexpr int kRB = kWK * 2;              // bytes per LDS row
constexpr int kVPR = kWK / 8;             // 16-byte vectors per row
constexpr int kRPB = 1024 / kRB;          // rows per 1 KB DMA block
// Token fragments per wave: 2 (16 waves, 64 x 64 per wave) and 4 (8 waves,
// 128 x 64, a quarter fewer LDS operand reads per MFMA) measured the same,
// so LDS bandwidth does not bound them either.
#ifndef EAT_WIDE_TF
#define EAT_WIDE_TF 2
#endif
constexpr int kTF = EAT_WIDE_TF;          // 32-row token fragments per wave
constexpr int kWaves = 4 * kWM / (32 * kTF);   // token groups x 4 weight quarters
constexpr int kThreads = kWaves * kWave;
constexpr int kRegion = kWM * kRB;        // bytes of one operand's rows per stage
constexpr int kStage = 2 * kRegion;       // tokens then weights
#ifndef EAT_WIDE_RING_KB
#define EAT_WIDE_RING_KB 128
#endif
constexpr int kStages = (EAT_WIDE_RING_KB * 1024) / kStage;   // ring depth
static_assert(kWN * kWK * 2 == kRegion, "token and weight regions have the same size");

struct WideArgs {
    const uint16_t* wa;        // [groups][M][K]  (W1, or W2 for the plain projection)
    const uint16_t* wb;        // [groups][M][K]  (W3, gated only)
    const uint16_t* src;       // activation rows, K wide
    const int32_t* gather;     // row -> source row, or null (identity)
    const int32_t* offsets;    // [groups+1] expert-major row offsets, or null
    int groups, nrows, M, K;
    void* out;                 // gated: bf16 H [rows][M]; plain: fp32 [rows][M] (bf16 with ROWS)
    float* nrm2;               // plain with ROWS: [rows][M / 32] sums of squares of 32 features of each row
    int xcds;                  // XCDs the grid is dealt over (the grid is a multiple of it)
};

// Byte offset of 16-byte vector v of row r in a region of kRB-byte rows.
// An MFMA operand read takes one vector of 16 consecutive rows per pass of
// the 64 LDS banks (256 bytes = kRowsPerLine rows); the XOR of the vector
// index with the row's line number spreads those 16 rows over distinct
// banks: (r >> 1) & 7 for 128-byte rows, (r >> 2) & 3 for 64-byte rows.
constexpr int kRowsPerLine = 256 / kRB;
// (unsigned: a signed division by the power of two costs a rounding fix-up
// and, in the wide kernel, the registers that then spill)
__device__ __forceinline__ int swz(int r) { return (static_cast<unsigned>(r) / kRowsPerLine) & (kVPR - 1); }
__device__ __forceinline__ int wswz(int r, int v) { return r * kRB + ((v ^ swz(r)) << 4); }

constexpr int kNB = (kWM + kWN) / kRPB;       // 1 KB DMA blocks per stage
constexpr int kBPW = kNB / kWaves;            // per wave
constexpr int kBT = kBPW / 2;                 // a wave's token blocks (the rest are weights)
constexpr int kP = kStages - 1;               // chunks in flight ahead of the one computed
static_assert(kNB % kWaves == 0, "blocks split evenly over the waves");
static_assert(kWM / kRPB == kWaves * kBT, "a wave's first half of blocks are token rows");
static_assert((kWN / 2) % kRPB == 0, "a DMA block holds rows of one gated matrix");
static_assert(kP <= 3, "wait counts cover up to three chunks in flight");

// One work item: token rows [r0, r0 + n) of expert e's segment against the
// expert's weight rows from m0 (W1 and W3 rows m0.. in the gated tile).
struct Item {
    int e, r0, n, m0;
};

// Lane l of a DMA instruction writes LDS bytes [16 l, 16 l + 16) of its 1 KB
// block = row l / kVPR, slot l % kVPR; it fetches the global vector that
// belongs in that slot under the swizzle.  Blocks j < kBT hold token rows (a
// 64-bit source per lane: rows are gathered), the others weight rows of
// expert e -- one matrix per block (W1 or W3 in the gated tile), so the
// block's base is uniform and each lane keeps a 32-bit element offset into
// the expert's matrix (M K < 2^31, checked on the host).
struct ItemLoads {
    const uint16_t* srct[kBT];
    uint32_t woff[kBPW - kBT];
    const uint16_t* wbase[kBPW - kBT];
};

// The source row of each of this lane's token blocks (rows past the expert's
// segment load a valid row; their results are unused).  Issued an item
// ahead, so the index loads complete under the previous item's chunks.
__device__ __forceinline__ void token_rows(const WideArgs& a, const Item& it, int (&srow)[kBT]) {
    const int lane = lane_id(), wave = threadIdx.x / kWave;
#pragma unroll
    for (int j = 0; j < kBT; ++j) {
        const int r = kRPB * (wave + kWaves * j) + lane / kVPR;
        const int g = r < it.n ? it.r0 + r : it.r0;
        srow[j] = a.gather ? a.gather[g] : g;
    }
}

template <bool GATED, bool PACKED>
__device__ __forceinline__ ItemLoads item_loads(const WideArgs& a, const Item& it, const int (&srow)[kBT]) {
    const int lane = lane_id(), wave = threadIdx.x / kWave;
    const int slot = lane % kVPR;
    ItemLoads L;
    const size_t emat = static_cast<size_t>(it.e) * a.M * a.K;
#pragma unroll
    for (int j = 0; j < kBPW; ++j) {
        const int b = wave + kWaves * j;
        if (j < kBT) {
            const int r = kRPB * b + lane / kVPR;
            const int v = slot ^ swz(r);
            L.srct[j] = a.src + static_cast<size_t>(srow[j]) * a.K + 8 * v;
        } else {
            const int rb0 = kRPB * (b - kWM / kRPB);          // the block's first weight row
            const int r = rb0 + lane / kVPR;
            const int v = slot ^ swz(r);
            const int row = it.m0 + (GATED ? (r & (kWN / 2 - 1)) : r);
            // packed: vector v of a chunk is k-step v / 4 of the chunk,
            // fragment (v % 4, row % 16) of that step's block (pack.hip)
            L.woff[j - kBT] = PACKED ? static_cast<uint32_t>(((row / 16) * (a.K / 32) + (v >> 2)) * 512 +
                                                             8 * (16 * (v & 3) + (row & 15)))
                                     : static_cast<uint32_t>(row * a.K + 8 * v);
            L.wbase[j - kBT] = (GATED && rb0 >= kWN / 2 ? a.wb : a.wa) + emat;
        }
    }
    return L;
}

// Chunk c of an item into LDS stage st.  asm keeps the compiler from adding
// waits of its own for these loads; the ring's waits and barriers order
// them.  Weight blocks load at device scope (sc1: no allocation in the CU's
// vector L1, which they would only churn -- a weight line is read once per
// workgroup); token rows keep the default policy.
template <bool PACKED>
__device__ __forceinline__ void issue_chunk(const ItemLoads& L, uint8_t* st, int c) {
    // elements a lane's source moves per chunk: token rows and row-major
    // weights by the chunk width, packed weights by its 512-element blocks
    constexpr int wstep = PACKED ? (kWK / 32) * 512 : kWK;
    const int wave = threadIdx.x / kWave;
#pragma unroll
    for (int j = 0; j < kBPW; ++j) {
        const uint16_t* src = j < kBT ? L.srct[j < kBT ? j : 0] + static_cast<size_t>(c) * kWK
                                      : L.wbase[j < kBT ? 0 : j - kBT] + L.woff[j < kBT ? 0 : j - kBT] +
                                            static_cast<size_t>(c) * wstep;
        const int b = wave + kWaves * j;
        const uint32_t lds = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(
            reinterpret_cast<uintptr_t>(st + (j < kBT ? 1024 * b : kRegion + 1024 * (b - kWM / kRPB)))));
        if (j < kBT)
            asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
                         :: "v"(src), "s"(lds) : "memory", "m0");
        else
            asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off sc1"
                         :: "v"(src), "s"(lds) : "memory", "m0");
    }
}

// Waits until at most `after` chunks' loads of this wave are still in flight
// (loads complete in issue order).
__device__ __forceinline__ void wait_chunks(int after) {
    if constexpr (kP >= 3) {
        if (after >= 2) wait_vm<2 * kBPW>();
        else if (after == 1) wait_vm<kBPW>();
        else wait_vm<0>();
    } else if constexpr (kP == 2) {
        if (after >= 1) wait_vm<kBPW>();
        else wait_vm<0>();
    } else {
        wait_vm<0>();
    }
}

// ROWS (plain tiles): the output rows are stored in bf16, and each lane
// writes the sum of squares of the 32 output features it holds of a row
// (half of its wave's 64), taken from the fp32 accumulators (the row norms
// of the account update).
template <bool GATED, bool PACKED, bool ROWS = false>
__global__ __launch_bounds__(kThreads) void wide_kernel(WideArgs a) {
    __shared__ __attribute__((aligned(1024))) uint8_t ring[kStages * kStage];
    __shared__ int tstart[kMaxExperts + 1];
    __shared__ int soff[kMaxExperts + 1];     // the segment offsets, read per item without a memory wait

    int ntiles;
    if (a.offsets) {
        for (int g = threadIdx.x; g <= a.groups; g += kThreads) soff[g] = a.offsets[g];
        tile_starts(a.offsets, a.groups, kWM, tstart);   // ends with a barrier
        ntiles = tstart[a.groups];
    } else {
        ntiles = (a.nrows + kWM - 1) / kWM;
    }
    constexpr int kOut = GATED ? kWN / 2 : kWN;     // output features per tile
    const int nx = a.M / kOut;
    const int work = ntiles * nx;
    const int xcd = blockIdx.x % a.xcds, slot = blockIdx.x / a.xcds;
    const int per_xcd = gridDim.x / a.xcds;
    const int part = (work + a.xcds - 1) / a.xcds;
    const int wbeg = xcd * part, wend = min(work, wbeg + part);

    // a workgroup's items only increase, so its segment search resumes where
    // the previous item's ended
    int es = 0;
    auto item_at = [&](int wid) __attribute__((always_inline)) {
        Item it;
        int tile = wid / nx, xt = wid % nx;
        if (a.offsets) {
            // an expert's items (the same range of wid as in tile-major
            // order) go weight tile by weight tile, its token tiles adjacent:
            // the workgroups that read one weight tile run in the same round,
            // even where the expert straddles a round of the XCD's slots
            while (tstart[es + 1] <= tile) ++es;
            const int nt = tstart[es + 1] - tstart[es];
            const int local = wid - tstart[es] * nx;
            xt = local / nt;
            tile = tstart[es] + local % nt;
            it.e = es;
            it.r0 = soff[es] + (tile - tstart[es]) * kWM;
            it.n = min(kWM, soff[es + 1] - it.r0);
        } else {
            it.e = 0;
            it.r0 = tile * kWM;
            it.n = min(kWM, a.nrows - it.r0);
        }
        it.m0 = xt * kOut;
        // uniform: keep the item in scalar registers
        it.e = __builtin_amdgcn_readfirstlane(it.e);
        it.r0 = __builtin_amdgcn_readfirstlane(it.r0);
        it.n = __builtin_amdgcn_readfirstlane(it.n);
        it.m0 = __builtin_amdgcn_readfirstlane(it.m0);
        return it;
    };

    int wid = wbeg + slot;
    if (wid >= wend) return;                  // uniform over the workgroup

    const int lane = lane_id(), wave = threadIdx.x / kWave;
    const int l32 = lane & 31, lh = lane >> 5;
    const int wm = wave >> 2, wn = wave & 3;  // token group, weight quarter (SIMD = wave % 4)
    const int brow = 32 * kTF * wm;           // this wave's first token row of the tile
    const int arow0 = GATED ? 32 * wn : 64 * wn;
    const int arow1 = GATED ? kWN / 2 + 32 * wn : 64 * wn + 32;
    const int nch = a.K / kWK;                // a multiple of kStages (K % 128 == 0)
    static_assert(128 % (kWK * kStages) == 0 || (kWK * kStages) % 128 == 0, "ring covers whole 128-wide steps");
    auto stage_of = [&](int c) __attribute__((always_inline)) { return ring + (c % kStages) * kStage; };

    // Ring of kStages stages, chunk c in stage c % kStages, loads issued kP
    // chunks ahead.  One step: wait for this wave's loads of chunk c (later
    // chunks' loads may stay in flight), barrier (every wave's loads of chunk
    // c have landed and every wave is done with chunk c - 1's stage), refill
    // that stage with chunk c + kP, compute chunk c.  The ring runs on across
    // items: an item's last steps issue the next item's first chunks (nch is a
    // multiple of kStages, so chunk c of every item sits in stage c % kStages),
    // and the next item's source rows are loaded an item ahead, so neither the
    // index loads nor the refill wait behind the item's output stores.
    Item cur = item_at(wid);
    int srow[kBT];
    token_rows(a, cur, srow);
    ItemLoads ld = item_loads<GATED, PACKED>(a, cur, srow);
#pragma unroll
    for (int c = 0; c < kP; ++c)
        if (c < nch) issue_chunk<PACKED>(ld, stage_of(c), c);

    for (;;) {
        const int nwid = wid + per_xcd;
        const bool more = nwid < wend;        // uniform
        Item nxt = cur;
        if (more) {
            nxt = item_at(nwid);
            token_rows(a, nxt, srow);
        }
        // this wave's token group holds rows of the expert (its fragments
        // past the tile's rows are skipped)
        const int ntf = min(kTF, max(0, (cur.n - brow + 31) / 32));
        const bool active = ntf > 0;
        f32x16 acc[2][kTF];                   // [weight fragment][token fragment]
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < kTF; ++j) acc[i][j] = f32x16{};

        // one step of the ring; L/ci: the loads to issue after the barrier
        // (ci < 0: none)
        auto step = [&](int c, const ItemLoads& L, int ci) __attribute__((always_inline)) {
            // chunks issued after c: the item's own, then the next item's
            // (the previous item's output stores may sit between them; a
            // wait that does not count them only waits longer)
            wait_chunks(more ? kP - 1 : min(kP - 1, nch - 1 - c));
            lds_barrier();
            if (ci >= 0) issue_chunk<PACKED>(L, stage_of(ci), ci);
            if (!active) return;
            const uint8_t* st = stage_of(c);
#pragma unroll
            for (int ks = 0; ks < kWK / 16; ++ks) {
                const int v = 2 * ks + lh;
                bf16x8 B[kTF], A[2];
#pragma unroll
                for (int j = 0; j < kTF; ++j)
                    B[j] = *reinterpret_cast<const bf16x8*>(st + wswz(brow + 32 * j + l32, v));
                A[0] = *reinterpret_cast<const bf16x8*>(st + kRegion + wswz(arow0 + l32, v));
                A[1] = *reinterpret_cast<const bf16x8*>(st + kRegion + wswz(arow1 + l32, v));
#pragma unroll
                for (int j = 0; j < kTF; ++j) {
                    if (kTF > 2 && j >= ntf) break;
#pragma unroll
                    for (int i = 0; i < 2; ++i)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A[i], B[j], acc[i][j], 0, 0, 0);
                }
            }
        };
        // steps that refill from this item, then (its loads all issued) the
        // last kP steps, which start the next item
        for (int c = 0; c + kP < nch; ++c) step(c, ld, c + kP);
        if (more) ld = item_loads<GATED, PACKED>(a, nxt, srow);
        for (int c = max(0, nch - kP); c < nch; ++c) step(c, ld, more ? c + kP - nch : -1);

        if (active) {
            // lane holds weight rows 8 (q / 4) + 4 lh + q % 4 of each 32-row
            // fragment, for token row brow + 32 j + l32
#pragma unroll
            for (int j = 0; j < kTF; ++j) {
                const int t = brow + 32 * j + l32;
                if (t >= cur.n) continue;
                const size_t orow = static_cast<size_t>(cur.r0 + t) * a.M;
                if constexpr (GATED) {
#pragma unroll
                    for (int qb = 0; qb < 4; ++qb) {
                        const int f = cur.m0 + 32 * wn + 8 * qb + 4 * lh;
                        uint16_t hv[4];
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            hv[q] = f32_to_bf16(silu(acc[0][j][4 * qb + q]) * acc[1][j][4 * qb + q]);
                        uint2 pk;
                        pk.x = static_cast<uint32_t>(hv[0]) | (static_cast<uint32_t>(hv[1]) << 16);
                        pk.y = static_cast<uint32_t>(hv[2]) | (static_cast<uint32_t>(hv[3]) << 16);
                        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.out) + orow + f) = pk;
                    }
                } else if constexpr (ROWS) {
                    float ss = 0.f;
#pragma unroll
                    for (int i = 0; i < 2; ++i)
#pragma unroll
                        for (int qb = 0; qb < 4; ++qb) {
                            const int f = cur.m0 + 64 * wn + 32 * i + 8 * qb + 4 * lh;
                            uint2 pk;
                            pk.x = pack_bf16x2(acc[i][j][4 * qb + 0], acc[i][j][4 * qb + 1]);
                            pk.y = pack_bf16x2(acc[i][j][4 * qb + 2], acc[i][j][4 * qb + 3]);
                            *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.out) + orow + f) = pk;
#pragma unroll
                            for (int q = 0; q < 4; ++q) ss = fmaf(acc[i][j][4 * qb + q], acc[i][j][4 * qb + q], ss);
                        }
                    // lanes l and l + 32 each hold half of the row's 64 features:
                    // slot m0 / 32 + 2 wn + lh of the row, whose slots start at
                    // r M / 32 = orow / 32 (from the first store's feature
                    // f0 = m0 + 64 wn + 4 lh, already at hand)
                    const int f0 = cur.m0 + 64 * wn + 4 * lh;
                    a.nrm2[(orow >> 5) + (f0 >> 5) + ((f0 >> 2) & 1)] = ss;
                } else {
#pragma unroll
                    for (int i = 0; i < 2; ++i)
#pragma unroll
                        for (int qb = 0; qb < 4; ++qb) {
                            const int f = cur.m0 + 64 * wn + 32 * i + 8 * qb + 4 * lh;
                            *reinterpret_cast<float4*>(static_cast<float*>(a.out) + orow + f) =
                                make_float4(acc[i][j][4 * qb + 0], acc[i][j][4 * qb + 1],
                                            acc[i][j][4 * qb + 2], acc[i][j][4 * qb + 3]);
                        }
                }
            }
        }
        if (!more) break;
        cur = nxt;
        wid = nwid;
    }
}

}  // namespace

bool wide_fits(bool gated, int M, int K) {
    return M % (gated ? kWN / 2 : kWN) == 0 && K % 128 == 0;
}

namespace {

// The part's geometry, asked once on the device current at the first call
// (every device a process uses is assumed to be the same part): workgroups
// of the wide kernel it keeps resident (one per CU: the ring takes 128 KB of
// LDS and the 16 waves fill the SIMDs) and the XCDs they are dealt over.
struct WideGeometry {
    int64_t resident;
    int xcds;
};

const WideGeometry& wide_geometry() {
    static const WideGeometry g = [] {
        int dev = 0, cus = 0, xccs = 0, per_cu = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
            cus = 256;
        if (hipDeviceGetAttribute(&xccs, hipDeviceAttributeNumberOfXccs, dev) != hipSuccess || xccs < 1 ||
            xccs > cus)
            xccs = 1;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, wide_kernel<true, true>, kThreads, 0) !=
                hipSuccess ||
            per_cu < 1)
            per_cu = 1;
        return WideGeometry{static_cast<int64_t>(cus) * per_cu, xccs};
    }();
    return g;
}

}  // namespace

hipError_t launch_wide(bool gated, const uint16_t* wa, const uint16_t* wb, const uint16_t* src,
                       const int32_t* gather, const int32_t* offsets, int groups, int nrows, int M, int K,
                       void* out, int64_t rows_cap, bool packed, float* nrm2, hipStream_t s) {
    if (nrm2 && gated) return hipErrorInvalidValue;
    const WideGeometry& geo = wide_geometry();
    WideArgs a{wa, wb, src, gather, offsets, groups, nrows, M, K, out, nrm2, geo.xcds};
    // every group may end in a partial tile
    const int64_t tiles = offsets ? std::min<int64_t>(rows_cap, (rows_cap + kWM - 1) / kWM + groups)
                                  : (nrows + kWM - 1) / kWM;
    const int64_t work = tiles * (M / (gated ? kWN / 2 : kWN));
    // persistent: the workgroups the part keeps resident (or one per item),
    // a multiple of the XCD count
    int64_t blocks = std::min<int64_t>(work, geo.resident);
    blocks = std::max<int64_t>(geo.xcds, (blocks + geo.xcds - 1) / geo.xcds * geo.xcds);
    const int nb = static_cast<int>(blocks);
    if (gated && packed) wide_kernel<true, true><<<nb, kThreads, 0, s>>>(a);
    else if (gated) wide_kernel<true, false><<<nb, kThreads, 0, s>>>(a);
    else if (nrm2 && packed) wide_kernel<false, true, true><<<nb, kThreads, 0, s>>>(a);
    else if (nrm2) wide_kernel<false, false, true><<<nb, kThreads, 0, s>>>(a);
    else if (packed) wide_kernel<false, true><<<nb, kThreads, 0, s>>>(a);
    else wide_kernel<false, false><<<nb, kThreads, 0, s>>>(a);
    return hipGetLastError();
}

}  // namespace eat
