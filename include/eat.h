/*
 * eat.h - C ABI of the EAT (Expert Account Tracker) MoE-layer forward for
 * AMD Instinct MI355X (gfx950).
 *
 * The library computes one Mixture-of-Experts layer forward with the
 * history-aware dynamic routing of "EAT: Expert Account Tracker for
 * Efficient MoE Inference" (Sec. 3), with fixed Top-K and Top-P routing as
 * switchable baselines:
 *
 *   router scores + softmax ............................ Sec. 3.1
 *   account statistics N, P_total, C_s; history score
 *     S_h (Eq. 1) and final importance I (Eq. 2) ........ Sec. 3.2
 *   adaptive threshold: grounding (Eq. 3-5), perplexity
 *     adjustment, boundedness, smoothing ................ Sec. 3.3
 *   activation set (Eq. 6), mask + renormalisation
 *     (Eq. 7-8), weighted fusion of expert outputs ...... Sec. 3.4
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Ownership: the caller owns every device buffer, including the account
 *    state and the workspace.  No call allocates device memory; the only
 *    device memory of the library's own is the fixed array that
 *    eat_moe_forward_noalloc uses in place of a workspace.
 *  - Asynchrony: every call that takes a stream only enqueues kernels on it
 *    and returns; inputs must stay alive and unmodified until the stream
 *    has passed the enqueued work.  No call synchronises the device.
 *  - Validation: all arguments are checked on the host before anything is
 *    enqueued.  On any error status nothing is launched and no output,
 *    workspace byte or account value is touched.
 *  - Errors: no C++ exception crosses this interface.  A HIP launch failure
 *    is reported as EAT_ERR_HIP (the enqueued work up to the failure may
 *    have run).
 *  - Limits: 1 <= E <= 256 (a token's mask is up to four 64-bit words);
 *    1 <= top_k <= E; d_model, d_ffn and d_shared are multiples of 64, with
 *    d_model * max(d_ffn, d_shared) < 2^31 elements per expert matrix;
 *    activations and expert weights are both fp32 or both bf16.
 *  - Layouts (all row-major, densely packed, 16-byte aligned; the expert
 *    weights may instead be packed, see eat_layout_t):
 *      x        [T][d_model]            act_dtype
 *      w_router [E][d_model]            fp32
 *      w1, w3   [E][d_ffn][d_model]     expert_dtype  (gate / up rows)
 *      w2       [E][d_model][d_ffn]     expert_dtype  (down rows)
 *      ws1, ws3 [d_shared][d_model], ws2 [d_model][d_shared]
 *      y        [T][d_model]            act_dtype
 *      masks    [T][W] uint64 with W = ceil(E / 64) words per token
 *               (one word for E <= 64): bit i % 64 of word i / 64 set
 *               <=> expert i selected
 *      gates    [T][E] fp32, renormalised gate (0 for unselected experts)
 *  - Non-finite inputs: a token whose row holds NaN or +-Inf gets NaN router
 *    scores; EAT then selects no expert for it, Top-K the K lowest-index
 *    experts, Top-P every expert up to top_p_cap; the other tokens of the
 *    call are unaffected.
 *  - Thread safety: a handle is immutable after eat_create; calls that use
 *    different workspaces and account buffers may run concurrently.
 *    Calls sharing an account buffer must be ordered on one stream.
 */
#ifndef EAT_H
#define EAT_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    EAT_OK = 0,
    EAT_ERR_INVALID_ARG = 1,   /* null / misaligned pointer, bad size or value */
    EAT_ERR_UNSUPPORTED = 2,   /* a shape or dtype outside the limits above   */
    EAT_ERR_WORKSPACE = 3,     /* workspace missing or smaller than required  */
    EAT_ERR_HIP = 4,           /* a HIP runtime call or kernel launch failed  */
    EAT_ERR_INTERNAL = 5,
    EAT_ERR_SCRATCH_LIMIT = 6  /* eat_moe_forward_noalloc: the call needs more
                                  than EAT_NOALLOC_SCRATCH_BYTES              */
} eat_status_t;

typedef enum {
    EAT_MODE_EAT = 0,          /* history-aware adaptive threshold (Sec. 3.2-3.4) */
    EAT_MODE_TOPK = 1,         /* vanilla Top-K (Sec. 3.1)                        */
    EAT_MODE_TOPP = 2          /* Top-P nucleus baseline (Sec. 4.1)               */
} eat_mode_t;

typedef enum { EAT_F32 = 0, EAT_BF16 = 1 } eat_dtype_t;

/* Layout of the bf16 expert weights w1, w3, w2 (and ws1, ws3, ws2).
 * ROWS: row-major as in the file header.  PACKED: the form eat_pack_weights
 * writes -- each matrix [groups][M][K] as 1 KB blocks of 16 rows x 32
 * reduction elements (block (g, r, s) at index (g M / 16 + r) K / 32 + s,
 * lane order of the matrix-core operand inside a block), which the decode
 * kernels read one contiguous kilobyte per load instruction. */
typedef enum { EAT_LAYOUT_ROWS = 0, EAT_LAYOUT_PACKED = 1 } eat_layout_t;

/* Layer shape and routing hyper-parameters.  eat_params_default() fills the
 * values of the paper's hyper-parameter table (Sec. 4.1) and the constants
 * of Sec. 3.3 / Eq. 7; the caller then sets the shape fields. */
typedef struct {
    int32_t mode;            /* eat_mode_t                                          */
    int32_t E;               /* routed experts, 1..256                              */
    int32_t d_model;         /* hidden width d                                      */
    int32_t d_ffn;           /* expert FFN width F                                  */
    int32_t top_k;           /* K: EAT's cap (Eq. 6) and Top-K's k; default 2       */
    float top_p;             /* Top-P threshold in (0, 1]; default 0.6              */
    int32_t top_p_cap;       /* 0 = uncapped nucleus, else max experts per token    */
    float alpha;             /* EMA factor of C_s (Sec. 3.2); 0.95                  */
    float w1, w2, w3;        /* Eq. 1 weights; 0.3, 0.3, 0.4                        */
    float beta;              /* Eq. 2 balance; 0.6                                  */
    float alpha1, alpha2;    /* Eq. 5 scaling; 0.5, 1.0                             */
    float kappa1, kappa2;    /* smoothing weights (Sec. 3.3); 0.7, 0.3              */
    float ppl_up, ppl_down;  /* tau factor when perplexity rose / otherwise; 1.2, 0.9 */
    float q_lo, q_hi;        /* bounds: these points of each token's routing
                                weights (linear interpolation, h = q (E-1)); 0.1, 0.9 */
    float eps;               /* Eq. 7 epsilon; 1e-8                                 */
    float inv_temperature;   /* router logits are multiplied by this; 1.0           */
    int32_t cs_mode;         /* 0: C_s enters Eq. 1 as is; 1: as C_s,i / sum C_s    */
    int32_t act_dtype;       /* eat_dtype_t of x and y                              */
    int32_t expert_dtype;    /* eat_dtype_t of w1/w3/w2 (and ws1/ws3/ws2)           */
    int32_t d_shared;        /* width of an always-on shared SwiGLU expert, 0 = none */
    const float* expert_scale; /* OPD reweighting (Sec. 3.5): device [E] fp32 scales s,
                                  p_i -> s_i p_i / sum_j s_j p_j before everything that
                                  uses p (importance, threshold, selection, gates,
                                  P_total), in every mode; NULL (default) = none.  The
                                  pointer is kept by eat_create and must stay valid,
                                  with s_i >= 0 and sum_j s_j p_j > 0, while the handle
                                  is used; 4-byte aligned.                          */
    int32_t weight_layout;   /* eat_layout_t of the expert weights; ROWS (default).
                                PACKED needs bf16 experts (UNSUPPORTED otherwise). */
} eat_params_t;

/* Per-layer account state (Sec. 3.2), device memory, length E each, owned by
 * the caller: activation counts N (int64), total gating probability P_total
 * (fp32) and the smoothed contribution C_s (fp32).  The state persists
 * across calls until eat_reset_accounts. */
typedef struct {
    int64_t* n;
    float* p_total;
    float* c_s;
} eat_accounts_t;

typedef struct eat_ctx* eat_handle_t;

/* Fill *out with the default hyper-parameters (mode EAT, E = 8,
 * d_model = 4096, d_ffn = 14336, bf16).  Returns EAT_ERR_INVALID_ARG for
 * a null pointer. */
eat_status_t eat_params_default(eat_params_t* out);

/* Validate params and build a handle for up to max_tokens tokens per call.
 * Host-only: no HIP call, no device memory.  Errors: INVALID_ARG for a null
 * pointer, a non-finite or out-of-range hyper-parameter or max_tokens
 * outside [1, 2^24]; UNSUPPORTED for a shape or dtype outside the limits in
 * the file header, or when max_tokens times the most experts a token can
 * select (top_k in Top-K, top_p_cap in capped Top-P, E otherwise) reaches
 * 2^31 (selected rows are indexed with 32-bit integers). */
eat_status_t eat_create(const eat_params_t* params, int32_t max_tokens, eat_handle_t* out);

/* Release a handle (host memory only).  Null is accepted. */
eat_status_t eat_destroy(eat_handle_t h);

/* Bytes of device workspace a call with T tokens needs (0 <= T <=
 * max_tokens).  The workspace holds router probabilities, gates, masks,
 * the token permutation and the expert intermediates, including the fp32
 * partial sums of projections whose reduction dimension is split (the
 * number of slices depends on T); it scales with T and is sized for the
 * mode's largest possible number of (token, expert) assignments (T*K for
 * Top-K, T*E for EAT and uncapped Top-P, since Eq. 6 keeps exact ties and
 * the nucleus is unbounded).  It is not monotonic in T: fewer tokens can
 * mean more slices (e.g. the Mixtral-shaped EAT layer needs more at T = 128
 * than at T = 129), so size a reused workspace by the largest value over the
 * T a caller will pass. */
eat_status_t eat_workspace_size(eat_handle_t h, int32_t T, size_t* bytes);

/* Zero the account state N, P_total, C_s (Sec. 3.2: the statistics start
 * empty) with a kernel on `stream` (no memset node, so it can be captured
 * in a graph). */
eat_status_t eat_reset_accounts(eat_handle_t h, eat_accounts_t acc, hipStream_t stream);

/* Bytes of device workspace eat_route needs for T tokens (the partial router
 * scores of its d slices).  Always <= eat_workspace_size(h, T), so a
 * forward workspace also serves routing. */
eat_status_t eat_route_workspace_size(eat_handle_t h, int32_t T, size_t* bytes);

/* Routing only (Sec. 3.1-3.4, no experts, accounts read but not updated).
 *   x          [T][d_model] act_dtype, device
 *   w_router   [E][d_model] fp32, device
 *   acc        account snapshot every token is judged against (EAT mode;
 *              ignored by Top-K / Top-P, may then hold null pointers)
 *   ppl_trend  [T] int8 or NULL: > 0 means the perplexity rose for that
 *              token's sequence (tau x ppl_up), anything else tau x ppl_down
 *   mask_out   [T][W] uint64 (W = ceil(E / 64)), k_out [T] int32,
 *              gate_out [T][E] fp32: required
 *   prob_out   [T][E] fp32 router probabilities, or NULL
 *   ws         device workspace of at least eat_route_workspace_size(h, T)
 *              bytes, 256-byte aligned (EAT_ERR_WORKSPACE otherwise)
 */
eat_status_t eat_route(eat_handle_t h, const void* x, int32_t T, const float* w_router,
                       eat_accounts_t acc, const int8_t* ppl_trend,
                       uint64_t* mask_out, int32_t* k_out, float* gate_out, float* prob_out,
                       void* ws, size_t ws_bytes, hipStream_t stream);

/* Whole layer forward over T tokens:
 *   y_t = sum over selected e of g_norm,t,e * SwiGLU_e(x_t)  (+ SwiGLU_shared(x_t))
 * with SwiGLU_e(x) = W2_e (silu(W1_e x) * (W3_e x)), no biases.
 * Every token routes against the accounts as they are when the call
 * starts; in EAT mode the accounts are then updated in place once for the
 * whole call (N += tokens routed to each expert, P_total += their router
 * probabilities, C_s <- (1 - alpha) C_s + alpha * mean ||o||_2 of the
 * expert's un-gated outputs); experts no token chose keep their values.
 * Top-K / Top-P neither read nor write the accounts.
 *   w1, w3, w2     routed experts (layouts in the file header)
 *   ws1, ws3, ws2  shared expert when d_shared > 0, else all NULL
 *   y              [T][d_model] act_dtype output
 *   mask_out       [T][W] uint64 (W = ceil(E / 64)) or NULL
 *   expert_load_out [E] int32 tokens per expert, or NULL
 */
eat_status_t eat_moe_forward(eat_handle_t h, const void* x, int32_t T, const float* w_router,
                             const void* w1, const void* w3, const void* w2,
                             const void* ws1, const void* ws3, const void* ws2,
                             eat_accounts_t acc, const int8_t* ppl_trend, void* y,
                             uint64_t* mask_out, int32_t* expert_load_out,
                             void* ws, size_t ws_bytes, hipStream_t stream);

/* Stage boundaries of eat_moe_forward, in launch order. */
typedef enum {
    EAT_STAGE_BEGIN = 0,      /* before routing                              */
    EAT_STAGE_ROUTED = 1,     /* routing done, before the permutation        */
    EAT_STAGE_PERMUTED = 2,   /* before the expert up/gate projection        */
    EAT_STAGE_UP = 3,         /* up/gate done, before the down projection    */
    EAT_STAGE_DOWN = 4,       /* down done, before the shared expert         */
    EAT_STAGE_SHARED = 5,     /* before the combine                          */
    EAT_STAGE_COMBINED = 6,   /* before the account update                   */
    EAT_STAGE_END = 7,        /* after the last kernel                       */
    EAT_NUM_STAGE_EVENTS = 8
} eat_stage_t;

/* eat_moe_forward that also records events[i] on `stream` at stage boundary
 * i for every non-null events[i], i < n_events <= EAT_NUM_STAGE_EVENTS, so a
 * caller can time individual kernels with hipEventElapsedTime.  Events are
 * created and owned by the caller.  Errors as eat_moe_forward; n_events
 * outside [0, EAT_NUM_STAGE_EVENTS] or a null array with n_events > 0 is
 * EAT_ERR_INVALID_ARG. */
eat_status_t eat_moe_forward_profiled(eat_handle_t h, const void* x, int32_t T, const float* w_router,
                                      const void* w1, const void* w3, const void* w2,
                                      const void* ws1, const void* ws3, const void* ws2,
                                      eat_accounts_t acc, const int8_t* ppl_trend, void* y,
                                      uint64_t* mask_out, int32_t* expert_load_out,
                                      void* ws, size_t ws_bytes, hipStream_t stream,
                                      const hipEvent_t* events, int32_t n_events);

/* ---- stacked layers -------------------------------------------------------
 *
 * The paper applies EAT in every MoE layer of a model, each layer keeping
 * its own account statistics (Sec. 3.2: the accounts are per expert of a
 * layer; Sec. 4 evaluates whole models).  eat_stack_forward runs one decode
 * step through n stacked MoE layers the way a decoder interleaves them with
 * its other blocks, here a normalisation and a residual mixing matrix:
 *
 *   u_l     = bf16( h_l / sqrt(mean_j h_l[j]^2 + rms_eps) )     (RMSNorm, unit gain)
 *   r_l     = bf16( h_l + MoE_l(u_l) )                          (layer l's forward)
 *   h_{l+1} = bf16( r_l . M_l^T )                               (fp32 accumulation)
 *
 * with h_0 = x and h_n written to h_out.  MoE_l is exactly eat_moe_forward
 * with layer l's handle, weights and accounts (which it reads and updates).
 * All layers need bf16 activations and experts and the same d_model. */
typedef struct {
    eat_handle_t layer;        /* the layer's handle (its mode, E, d_ffn, K, ...)        */
    const float* w_router;     /* [E][d] fp32                                            */
    const void* w1;            /* [E][F][d] bf16                                         */
    const void* w3;            /* [E][F][d] bf16                                         */
    const void* w2;            /* [E][d][F] bf16                                         */
    const void* ws1;           /* always-on expert [F_sh][d], [F_sh][d], [d][F_sh] bf16, */
    const void* ws3;           /*   or NULL when the layer declares none                 */
    const void* ws2;
    const void* mix;           /* [d][d] bf16 mixing matrix M_l (row-major, M_l[out][in]) */
    eat_accounts_t acc;        /* layer l's account state (EAT mode)                     */
} eat_stack_layer_t;

/* Workspace bytes eat_stack_forward needs for T tokens through `layers`
 * (host array of n_layers entries).  Errors: EAT_ERR_INVALID_ARG (null
 * pointers, n_layers outside [1, 1024], T < 0 or above a layer's max_tokens,
 * different d_model, a null or misaligned mix), EAT_ERR_UNSUPPORTED (a layer
 * that is not bf16, or d_model not a multiple of 8 or above 8192). */
eat_status_t eat_stack_workspace_size(const eat_stack_layer_t* layers, int32_t n_layers, int32_t T,
                                      size_t* bytes);

/* One step of T tokens through the stacked layers (formulas above).
 *   layers     host array [n_layers]; device pointers inside, 16-byte aligned
 *   x          [T][d] bf16 input h_0 (device, read only)
 *   ppl_trend  [T] int8 or NULL, passed to every layer (Sec. 3.3)
 *   rms_eps    RMSNorm epsilon (finite, >= 0)
 *   h_out      [T][d] bf16 output h_n (device; must not alias x)
 *   masks_out  every layer's selection masks, layer after layer,
 *              [T][ceil(E_l / 64)] uint64 each, or NULL
 *   probs_out  every layer's router probabilities p (Sec. 3.1), layer after
 *              layer, [T][E_l] fp32 each (T * sum of E_l floats), or NULL
 *   ws         device workspace of eat_stack_workspace_size bytes, 256-byte aligned
 * Enqueues on `stream` only; no host synchronisation, no allocation.  Every
 * layer's accounts are updated as its eat_moe_forward would (EAT mode).
 * Errors: as eat_stack_workspace_size and eat_moe_forward, checked on the
 * host before anything is enqueued; EAT_ERR_HIP if a launch fails. */
eat_status_t eat_stack_forward(const eat_stack_layer_t* layers, int32_t n_layers, const void* x, int32_t T,
                               const int8_t* ppl_trend, float rms_eps, void* h_out, uint64_t* masks_out,
                               float* probs_out, void* ws, size_t ws_bytes, hipStream_t stream);

/* ---- perplexity signal ----------------------------------------------------
 *
 * Sec. 3.3 raises the threshold by 20% when the model's perplexity rose
 * (PPL_curr - PPL_prev > 0) and lowers it by 10% otherwise.  eat_ppl_trend
 * produces that signal for S sequences, one token each, from the LM head:
 *
 *   z_s   = h_s . W_V^T                      (bf16 in, fp32 accumulation)
 *   NLL_s = logsumexp(z_s) - z_s[target_s]
 *   sum_s += NLL_s;  n_s += 1;  PPL_s = exp(sum_s / n_s)        (fp64 state)
 *   trend_s = +1 if n_s > 1 and PPL_s > PPL_prev_s, -1 if n_s > 1 otherwise,
 *             0 for a sequence's first token;  PPL_prev_s = PPL_s
 *
 * trend_out is the int8 ppl_trend the next step's eat_route /
 * eat_moe_forward / eat_stack_forward take for those sequences' tokens. */

/* Workspace bytes for S sequences, width d (multiple of 64) and vocabulary
 * V (multiple of 64), d * V < 2^31.  EAT_ERR_INVALID_ARG otherwise. */
eat_status_t eat_ppl_workspace_size(int32_t S, int32_t d, int32_t V, size_t* bytes);

/* Zero the running state of S sequences (device arrays, caller-owned):
 * nll_sum [S] fp64, count [S] int32, ppl_prev [S] fp64. */
eat_status_t eat_ppl_reset(int32_t S, double* nll_sum, int32_t* count, double* ppl_prev, hipStream_t stream);

/* One token per sequence through the LM head (formulas above).
 *   h          [S][d] bf16 final hidden rows (device)
 *   w_vocab    [V][d] bf16 LM head (device)
 *   target     [S] int32 next-token ids; an id outside [0, V) gives a NaN
 *              NLL and a NaN running sum for that sequence, whose trend
 *              is then -1 until eat_ppl_reset (NaN compares false)
 *   nll_sum, count, ppl_prev   the running state, updated in place
 *   trend_out  [S] int8;  nll_out [S] fp32 or NULL
 *   ws         workspace of eat_ppl_workspace_size bytes, 256-byte aligned
 * Enqueues on `stream` only; no synchronisation, no allocation.  Errors:
 * EAT_ERR_INVALID_ARG (shapes, null or misaligned pointers),
 * EAT_ERR_WORKSPACE, EAT_ERR_HIP. */
eat_status_t eat_ppl_trend(const void* h, int32_t S, int32_t d, const void* w_vocab, int32_t V,
                           const int32_t* target, double* nll_sum, int32_t* count, double* ppl_prev,
                           int8_t* trend_out, float* nll_out, void* ws, size_t ws_bytes, hipStream_t stream);

/* ---- packed expert weights -------------------------------------------------
 *
 * Write the PACKED form (eat_layout_t) of `groups` row-major bf16 matrices
 * [groups][M][K] (device src) into dst (device, groups * M * K bf16, must not
 * overlap src); e.g. w1 as (E, d_ffn, d_model), w2 as (E, d_model, d_ffn),
 * ws1 as (1, d_shared, d_model).  M a multiple of 16, K of 32, both > 0;
 * groups >= 1; 16-byte aligned pointers.  A permutation: a layer created with
 * weight_layout = PACKED on the packed copies computes bit-identical results.
 * Enqueues on `stream` only.  Errors: EAT_ERR_INVALID_ARG, EAT_ERR_HIP. */
eat_status_t eat_pack_weights(const void* src, int32_t groups, int32_t M, int32_t K, void* dst,
                              hipStream_t stream);

/* ---- allocation-free forward -----------------------------------------------
 *
 * For callers that cannot allocate device memory at call time: code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation.
 * eat_moe_forward_noalloc is eat_moe_forward (same arguments, results
 * bit-identical to it) without the workspace arguments: its intermediates
 * live in a fixed device array of EAT_NOALLOC_SCRATCH_BYTES that the
 * library holds on every GPU it runs this entry point on, until the process
 * ends.  The caller still owns and passes every input, output and the
 * account state.  The call allocates and frees nothing; the array's device
 * address is looked up once per device, on the first call with that device
 * current (make that first call outside graph capture).
 *   Limit: a call whose eat_workspace_size(h, T) exceeds
 *   EAT_NOALLOC_SCRATCH_BYTES returns EAT_ERR_SCRATCH_LIMIT and enqueues
 *   nothing (e.g. the Mixtral-shaped EAT layer fits up to T = 64 tokens).
 *   Sharing: every call on one GPU uses that GPU's one array, and no part
 *   of it needs clearing (each call writes every byte it reads first), so
 *   consecutive calls are independent; calls whose executions overlap on
 *   one GPU (different streams without ordering, several host threads)
 *   race on the array and give undefined results: order them on one stream.
 * Errors: as eat_moe_forward, plus EAT_ERR_SCRATCH_LIMIT; EAT_ERR_HIP if the
 * device or the array's address cannot be obtained or a launch fails. */
#define EAT_NOALLOC_SCRATCH_BYTES ((size_t)256 << 20)

eat_status_t eat_moe_forward_noalloc(eat_handle_t h, const void* x, int32_t T, const float* w_router,
                                     const void* w1, const void* w3, const void* w2,
                                     const void* ws1, const void* ws3, const void* ws2,
                                     eat_accounts_t acc, const int8_t* ppl_trend, void* y,
                                     uint64_t* mask_out, int32_t* expert_load_out, hipStream_t stream);

/* Static description of a status code (never NULL). */
const char* eat_status_string(eat_status_t s);

#ifdef __cplusplus
}
#endif

#endif /* EAT_H */
