// Host-side internals of the EAT library: the validated handle, the
// workspace carve-up and the kernel launchers each .hip file provides.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <algorithm>
#include <functional>

#include "../../include/eat.h"

struct eat_ctx {
    eat_params_t p;
    int32_t max_tokens;
    int32_t kmax;            // largest possible experts per token in this mode
};

namespace eat {

constexpr int kMaxExperts = 256;   // selection masks of up to four 64-bit words per token

// 64-bit words of one token's selection mask: bit e % 64 of word e / 64 is expert e.
inline int mask_words(int E) { return (E + 63) / 64; }

// Offsets (bytes) of the workspace regions for T tokens.  Every region
// starts on a 256-byte boundary.
// Small values the kernels of one call hand to each other (workspace region
// `sync`, kSyncWords words): [0] the slices the routed up/gate projection
// took, [1] the slices the down projection took.
constexpr int kSyncWords = 2;

struct Workspace {
    size_t lpart, prob, gate, mask, k, offsets, tok_idx, inv, row_expert, h, gu, yp, nrm, hs, ys, gus, ysp, sync;
    size_t route_total;      // bytes eat_route needs (the leading lpart region)
    size_t total;
    int64_t rows;            // capacity in (token, expert) rows = T * kmax
    int splits;              // down-projection slices held in yp
    int up_splits;           // up/gate slices held in gu (1: gu unused)
    int shared_splits;       // always-on expert's down-projection slices held in ysp (1: ysp unused)
    int shared_up_splits;    // its up/gate slices held in gus (1: gus unused)
};
Workspace plan_workspace(const eat_ctx& c, int32_t T);

// Pointers into a workspace for one call.
struct Buffers {
    float* lpart;            // [route_slices][T][E] partial router scores
    float* prob;             // [T][E] router probabilities
    float* gate;             // [T][E] renormalised gates
    uint64_t* mask;          // [T][mask_words(E)]
    int32_t* k;              // [T]
    int32_t* offsets;        // [E+1] expert-major row offsets
    int32_t* tok_idx;        // [rows] token of each expert-major row
    int32_t* inv;            // [T][E] row of (t, e), valid where selected
    int32_t* row_expert;     // [rows] expert of each row
    void* h;                 // [rows][F] SwiGLU hidden (bf16 or fp32)
    float* gu;               // [2][up_splits][rows][F] gate / up partial sums
    float* yp;               // [splits][rows][d] un-gated expert outputs (partials)
    float* nrm2;             // [rows][norm_parts] partial sums of squares of yp rows
    void* hs;                // [T][F_sh] shared-expert hidden
    float* ys;               // [T][d] shared-expert output
    float* gus;              // [2][shared_up_splits][T][F_sh] its gate / up partial sums
    float* ysp;              // [shared_splits][T][d] its down-projection partial sums
    unsigned* sync;          // kSyncWords words (see above)
};

// ---- launchers (return hipGetLastError() after enqueueing) -------------

hipError_t launch_reset_accounts(const eat_params_t& p, eat_accounts_t acc, hipStream_t s);

// Routing: partial router scores per (token tile, d slice) into `part`
// ([route_slices][T][E] fp32), then one selection wave per token.
hipError_t launch_route(const eat_params_t& p, const void* x, int32_t T, const float* w_router,
                        eat_accounts_t acc, const int8_t* trend, float* part, uint64_t* mask, int32_t* k,
                        float* gate, float* prob, hipStream_t s);
int route_token_tiles(int32_t T);                  // 16-token MFMA tiles per logits workgroup
int route_slices(const eat_params_t& p, int32_t T);  // d slices of the logits kernel

hipError_t launch_permute(const eat_params_t& p, int32_t T, const uint64_t* mask,
                          int32_t* offsets, int32_t* tok_idx, int32_t* inv, int32_t* row_expert,
                          int32_t* expert_load, hipStream_t s);

// Routed experts.  `between` runs on the host after the up/gate launch and
// before the down launch (stage-event hook).
// fp32 weights and activations (small layers):
hipError_t launch_experts_f32(const eat_params_t& p, int32_t T, int64_t rows_cap, const float* x,
                              const float* w1, const float* w3, const float* w2,
                              const int32_t* offsets, const int32_t* tok_idx,
                              const int32_t* row_expert, float* h, float* yp, hipStream_t s,
                              const std::function<void()>& between);

// bf16 weights and activations: MFMA kernels.  Both projections choose
// their slices on the device and write the count they took to
// *up_splits_dev / *down_splits_dev (read by the up/gate slice reduce and
// by the combine).  When rows_bf16(p, T), yp receives bf16 rows and nrm2
// their partial sums of squares (norm_parts per row).
hipError_t launch_experts_bf16(const eat_params_t& p, int32_t T, int64_t rows_cap,
                               const uint16_t* x, const uint16_t* w1, const uint16_t* w3,
                               const uint16_t* w2, const int32_t* offsets, const int32_t* tok_idx,
                               uint16_t* h, float* gu, float* yp, float* nrm2, int32_t* up_splits_dev,
                               int32_t* down_splits_dev, hipStream_t s, const std::function<void()>& between);

// Always-on shared expert over all T tokens.
hipError_t launch_shared_f32(const eat_params_t& p, int32_t T, const float* x, const float* ws1,
                             const float* ws3, const float* ws2, float* hs, float* ys,
                             hipStream_t s);
// bf16: the reduction dimensions split into shared_up_splits / shared_splits
// slices (fp32 partials in gus / ysp, added in slice order) when the call is
// too small to fill the chip with whole rows.
int shared_up_splits(const eat_params_t& p, int32_t T);
int shared_splits(const eat_params_t& p, int32_t T);
hipError_t launch_shared_bf16(const eat_params_t& p, int32_t T, const uint16_t* x,
                              const uint16_t* ws1, const uint16_t* ws3, const uint16_t* ws2,
                              uint16_t* hs, float* ys, float* gus, float* ysp, hipStream_t s);

// yp holds the down projection's partial slices, `split_stride` floats
// apart (*splits_dev of them when set, else `splits`); they are added in
// slice order, and each row slice's sum of squares goes to nrm2.  With
// rows_bf16 yp holds bf16 rows instead (one slice) whose sums of squares
// are already in nrm2.  `residual` (bf16 [T][d], or null) is added to y
// before the cast.
hipError_t launch_combine(const eat_params_t& p, int32_t T, const uint64_t* mask,
                          const float* gate, const int32_t* inv, const void* yp,
                          const float* ys, const uint16_t* residual, void* y, float* nrm2,
                          int splits, int64_t split_stride, const int32_t* splits_dev, bool rows_bf16,
                          hipStream_t s);

// Between stacked layers (combine.hip): h = bf16(sum of `splits` fp32
// partial rows, or the bf16 rows of src when splits == 0), written to h_out
// if set; u = bf16(h / sqrt(mean(h^2) + eps)) written to u_out if set.
// `accounts` (or null): a deferred account update, done by extra
// workgroups of the same launch (it depends on neither h nor u).
struct AccountJob;
bool mix_norm_fits(int d);
hipError_t launch_mix_norm(const float* part, int splits, int64_t split_stride, const uint16_t* src,
                           int32_t T, int d, float eps, uint16_t* h_out, uint16_t* u_out,
                           const AccountJob* accounts, hipStream_t s);

// Dense bf16 projection out[split][T][M] = src[T][K] . W^T (fp32 slices of
// the reduction dimension, split_stride floats apart), W [M][K]: the
// residual mixing of stacked layers (expert.hip).
int dense_splits(int M, int K, int32_t T);
hipError_t launch_dense_bf16(const uint16_t* src, int32_t T, const uint16_t* w, int M, int K, float* out,
                             int splits, int64_t split_stride, hipStream_t s);
// 1024-element slices of d the combine works in.
int combine_chunks(const eat_params_t& p);
// Prefill-sized bf16 calls: the down projection (wide tiles) stores the
// expert rows of yp in bf16 with their norms' partial sums of squares, one
// per 32 features (expert.hip); other calls keep fp32 rows whose sums of
// squares the combine takes, one per combine chunk.
bool rows_bf16(const eat_params_t& p, int32_t T);
// Partial sums of squares per expert row in nrm2.
int norm_parts(const eat_params_t& p, int32_t T);

// Number of reduction-dimension slices the bf16 down projection uses for T
// tokens (1 for fp32 layers).
int down_splits(const eat_params_t& p, int32_t T);
// Slices of the bf16 up/gate projection; above 1 the gate and up sums go
// through fp32 partial buffers (workspace region gu) and a reduce kernel.
int up_splits(const eat_params_t& p, int32_t T);

// Grouped bf16 GEMM with 256 x 256 tiles for prefill-sized calls (wide.hip):
// gated = H = bf16(silu(x W1^T) * (x W3^T)) over 128-feature tiles, plain =
// fp32 out = src W^T over 256-row tiles.  Rows are the expert segments given
// by offsets (gather maps them to source rows), or nrows identity rows when
// offsets is null.  wide_fits tells whether M and K suit the tiling; `packed`
// reads wa / wb in the packed layout.  With nrm2 (plain tiles) out holds
// bf16 rows and nrm2 [rows][M / 32] partial sums of squares of each row (32
// features each), taken before the cast.
bool wide_fits(bool gated, int M, int K);
hipError_t launch_wide(bool gated, const uint16_t* wa, const uint16_t* wb, const uint16_t* src,
                       const int32_t* gather, const int32_t* offsets, int groups, int nrows, int M,
                       int K, void* out, int64_t rows_cap, bool packed, float* nrm2, hipStream_t s);

// Packed weight layout (pack.hip): dst = the 1 KB-block form of the
// row-major bf16 [groups][M][K] src (M % 16 == 0, K % 32 == 0).
hipError_t launch_pack(const uint16_t* src, int32_t groups, int32_t M, int32_t K, uint16_t* dst, hipStream_t s);

// Perplexity signal (ppl.hip): z [S][V] fp32 LM-head rows -> NLL of target,
// running per-sequence state (fp64 NLL sum, count, previous perplexity) and
// the int8 trend; z holds `splits` slices `stride` floats apart.
// launch_ppl_reset zeroes the state.
hipError_t launch_ppl(const float* z, int splits, int64_t stride, int32_t S, int V, const int32_t* target,
                      double* nll_sum, int32_t* count, double* ppl_prev, int8_t* trend, float* nll_out,
                      float2* part, hipStream_t s);
int ppl_splits(int32_t S, int d, int V);
int ppl_chunks(int V);                 // (max, sum) pairs per row in `part`
hipError_t launch_ppl_reset(int32_t S, double* nll_sum, int32_t* count, double* ppl_prev, hipStream_t s);

// Forward entry points (api.cpp): host-side argument checks, and the
// enqueue of one layer forward into a workspace of plan_workspace(h, T).total
// bytes at `ws` (arguments checked, T > 0).  `residual` (bf16 [T][d] or
// null) is added to y; `prob_out` (or null) receives the router probabilities.
eat_status_t check_forward(const eat_ctx* h, const void* x, int32_t T, const float* w_router, const void* w1,
                           const void* w3, const void* w2, const void* ws1, const void* ws3, const void* ws2,
                           const eat_accounts_t& acc, const void* y, const uint64_t* mask_out,
                           const int32_t* expert_load_out);
// The account update of one call (Sec. 3.2): its inputs in the call's
// workspace, and the accounts.  experts == 0: nothing to update (baseline
// modes, or no call).
struct AccountJob {
    const int32_t* offsets;
    const int32_t* tok_idx;
    const float* prob;
    const float* nrm2;
    int parts;               // partial sums of squares per row in nrm2
    int experts;
    float alpha;
    eat_accounts_t acc;
};
// With `defer` set, the account update is not enqueued but described there,
// for a later launch on the same stream (before the workspace is reused).
hipError_t forward_impl(const eat_ctx& h, const void* x, int32_t T, const float* w_router, const void* w1,
                        const void* w3, const void* w2, const void* ws1, const void* ws3, const void* ws2,
                        eat_accounts_t acc, const int8_t* ppl_trend, const uint16_t* residual, void* y,
                        uint64_t* mask_out, int32_t* expert_load_out, float* prob_out, void* ws,
                        hipStream_t stream, const hipEvent_t* events, int32_t n_events,
                        AccountJob* defer = nullptr);

// nrm2: `parts` partial sums of squares per row, added in order.
hipError_t launch_update_accounts(const eat_params_t& p, const int32_t* offsets,
                                  const int32_t* tok_idx, const float* prob, const float* nrm2, int parts,
                                  eat_accounts_t acc, hipStream_t s);

}  // namespace eat
