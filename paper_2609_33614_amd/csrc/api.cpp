// C ABI of the EAT MoE-layer library: argument validation, workspace
// carve-up and the launch sequence.  Every check runs on the host before
// any HIP call; no exception leaves this file.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <cstring>
#include <cmath>
#include <functional>
#include <new>

#include "eat_internal.h"

namespace {

constexpr int32_t kMaxTokens = 1 << 24;

bool finite(float v) { return isfinite(v) != 0; }
bool in01(float v) { return finite(v) && v >= 0.f && v <= 1.f; }
bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

eat_status_t check_params(const eat_params_t& p) {
    if (p.mode < EAT_MODE_EAT || p.mode > EAT_MODE_TOPP) return EAT_ERR_INVALID_ARG;
    if (p.E < 1 || p.d_model < 1 || p.d_ffn < 1 || p.d_shared < 0) return EAT_ERR_INVALID_ARG;
    if (p.top_k < 1 || p.top_k > p.E) return EAT_ERR_INVALID_ARG;
    if (p.mode == EAT_MODE_TOPP && !(finite(p.top_p) && p.top_p > 0.f && p.top_p <= 1.f))
        return EAT_ERR_INVALID_ARG;
    if (p.top_p_cap < 0 || p.top_p_cap > p.E) return EAT_ERR_INVALID_ARG;
    if (!in01(p.alpha) || !in01(p.beta)) return EAT_ERR_INVALID_ARG;
    const float fin[] = {p.w1, p.w2, p.w3, p.alpha1, p.alpha2, p.kappa1, p.kappa2,
                         p.ppl_up, p.ppl_down, p.eps, p.inv_temperature};
    for (float v : fin)
        if (!finite(v)) return EAT_ERR_INVALID_ARG;
    if (!in01(p.q_lo) || !in01(p.q_hi) || p.q_lo > p.q_hi) return EAT_ERR_INVALID_ARG;
    if (p.eps < 0.f || p.inv_temperature <= 0.f) return EAT_ERR_INVALID_ARG;
    if (p.cs_mode != 0 && p.cs_mode != 1) return EAT_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(p.expert_scale) % 4) return EAT_ERR_INVALID_ARG;
    if ((p.act_dtype != EAT_F32 && p.act_dtype != EAT_BF16) ||
        (p.expert_dtype != EAT_F32 && p.expert_dtype != EAT_BF16))
        return EAT_ERR_INVALID_ARG;
    // supported shapes and dtype pairs
    if (p.E > eat::kMaxExperts) return EAT_ERR_UNSUPPORTED;
    if (p.d_model % 64 || p.d_ffn % 64 || p.d_shared % 64) return EAT_ERR_UNSUPPORTED;
    // one expert matrix is addressed with 32-bit element offsets
    if (static_cast<int64_t>(p.d_model) * std::max(p.d_ffn, p.d_shared) >= (int64_t{1} << 31))
        return EAT_ERR_UNSUPPORTED;
    if (p.act_dtype != p.expert_dtype) return EAT_ERR_UNSUPPORTED;
    if (p.weight_layout != EAT_LAYOUT_ROWS && p.weight_layout != EAT_LAYOUT_PACKED) return EAT_ERR_INVALID_ARG;
    if (p.weight_layout == EAT_LAYOUT_PACKED && p.expert_dtype != EAT_BF16) return EAT_ERR_UNSUPPORTED;
    return EAT_OK;
}

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

}  // namespace

namespace eat {

Workspace plan_workspace(const eat_ctx& c, int32_t T) {
    const eat_params_t& p = c.p;
    Workspace w{};
    const size_t t = static_cast<size_t>(T), E = static_cast<size_t>(p.E);
    const size_t es = p.expert_dtype == EAT_BF16 ? 2 : 4;
    w.rows = static_cast<int64_t>(T) * c.kmax;
    w.splits = down_splits(p, T);
    w.up_splits = up_splits(p, T);
    const size_t rows = static_cast<size_t>(w.rows);
    size_t off = 0;
    auto take = [&](size_t bytes) { const size_t at = off; off += align256(bytes); return at; };
    w.lpart = take(static_cast<size_t>(T > 0 ? route_slices(p, T) : 1) * t * E * 4);
    w.route_total = off;
    w.prob = take(t * E * 4);
    w.gate = take(t * E * 4);
    w.mask = take(t * eat::mask_words(p.E) * 8);
    w.k = take(t * 4);
    w.offsets = take((E + 1) * 4);
    w.tok_idx = take(rows * 4);
    w.inv = take(t * E * 4);
    w.row_expert = take(rows * 4);
    w.h = take(rows * p.d_ffn * es);
    w.gu = take(w.up_splits > 1 ? 2 * static_cast<size_t>(w.up_splits) * rows * p.d_ffn * 4 : 0);
    w.yp = take(static_cast<size_t>(w.splits) * rows * p.d_model * 4);
    w.nrm = take(rows * static_cast<size_t>(norm_parts(p, T)) * 4);
    w.shared_splits = p.d_shared ? shared_splits(p, T) : 1;
    w.shared_up_splits = p.d_shared ? shared_up_splits(p, T) : 1;
    w.hs = take(p.d_shared ? t * p.d_shared * es : 0);
    w.ys = take(p.d_shared ? t * p.d_model * 4 : 0);
    w.gus = take(w.shared_up_splits > 1 ? 2 * static_cast<size_t>(w.shared_up_splits) * t * p.d_shared * 4 : 0);
    w.ysp = take(w.shared_splits > 1 ? static_cast<size_t>(w.shared_splits) * t * p.d_model * 4 : 0);
    w.sync = take(static_cast<size_t>(kSyncWords) * 4);
    w.total = off;
    return w;
}

}  // namespace eat

extern "C" {

eat_status_t eat_params_default(eat_params_t* out) {
    if (!out) return EAT_ERR_INVALID_ARG;
    memset(out, 0, sizeof(*out));
    out->mode = EAT_MODE_EAT;
    out->E = 8;
    out->d_model = 4096;
    out->d_ffn = 14336;
    out->top_k = 2;
    out->top_p = 0.6f;
    out->top_p_cap = 0;
    out->alpha = 0.95f;
    out->w1 = 0.3f; out->w2 = 0.3f; out->w3 = 0.4f;
    out->beta = 0.6f;
    out->alpha1 = 0.5f; out->alpha2 = 1.0f;
    out->kappa1 = 0.7f; out->kappa2 = 0.3f;
    out->ppl_up = 1.2f; out->ppl_down = 0.9f;
    out->q_lo = 0.1f; out->q_hi = 0.9f;
    out->eps = 1e-8f;
    out->inv_temperature = 1.0f;
    out->cs_mode = 0;
    out->act_dtype = EAT_BF16;
    out->expert_dtype = EAT_BF16;
    out->d_shared = 0;
    out->expert_scale = nullptr;
    out->weight_layout = EAT_LAYOUT_ROWS;
    return EAT_OK;
}

eat_status_t eat_create(const eat_params_t* params, int32_t max_tokens, eat_handle_t* out) {
    if (!params || !out) return EAT_ERR_INVALID_ARG;
    *out = nullptr;
    if (max_tokens < 1 || max_tokens > kMaxTokens) return EAT_ERR_INVALID_ARG;
    const eat_status_t st = check_params(*params);
    if (st != EAT_OK) return st;
    // most (token, expert) rows a call can select: rows, segment offsets and
    // token indices are 32-bit
    int32_t kmax = params->E;
    if (params->mode == EAT_MODE_TOPK) kmax = params->top_k;
    else if (params->mode == EAT_MODE_TOPP && params->top_p_cap > 0) kmax = params->top_p_cap;
    if (static_cast<int64_t>(max_tokens) * kmax >= (int64_t{1} << 31)) return EAT_ERR_UNSUPPORTED;
    eat_ctx* c = new (std::nothrow) eat_ctx;
    if (!c) return EAT_ERR_INTERNAL;
    c->p = *params;
    c->max_tokens = max_tokens;
    c->kmax = kmax;
    *out = c;
    return EAT_OK;
}

eat_status_t eat_destroy(eat_handle_t h) {
    delete h;
    return EAT_OK;
}

eat_status_t eat_workspace_size(eat_handle_t h, int32_t T, size_t* bytes) {
    if (!h || !bytes || T < 0 || T > h->max_tokens) return EAT_ERR_INVALID_ARG;
    *bytes = eat::plan_workspace(*h, T).total;
    return EAT_OK;
}

eat_status_t eat_reset_accounts(eat_handle_t h, eat_accounts_t acc, hipStream_t stream) {
    if (!h || !acc.n || !acc.p_total || !acc.c_s) return EAT_ERR_INVALID_ARG;
    if (!aligned(acc.n, 8) || !aligned(acc.p_total, 4) || !aligned(acc.c_s, 4)) return EAT_ERR_INVALID_ARG;
    (void)hipGetLastError();
    return eat::launch_reset_accounts(h->p, acc, stream) == hipSuccess ? EAT_OK : EAT_ERR_HIP;
}

static eat_status_t check_accounts(const eat_ctx& c, const eat_accounts_t& acc) {
    if (c.p.mode != EAT_MODE_EAT) return EAT_OK;
    if (!acc.n || !acc.p_total || !acc.c_s) return EAT_ERR_INVALID_ARG;
    if (!aligned(acc.n, 8) || !aligned(acc.p_total, 4) || !aligned(acc.c_s, 4)) return EAT_ERR_INVALID_ARG;
    return EAT_OK;
}

eat_status_t eat_route_workspace_size(eat_handle_t h, int32_t T, size_t* bytes) {
    if (!h || !bytes || T < 0 || T > h->max_tokens) return EAT_ERR_INVALID_ARG;
    *bytes = eat::plan_workspace(*h, T).route_total;
    return EAT_OK;
}

eat_status_t eat_route(eat_handle_t h, const void* x, int32_t T, const float* w_router,
                       eat_accounts_t acc, const int8_t* ppl_trend, uint64_t* mask_out,
                       int32_t* k_out, float* gate_out, float* prob_out, void* ws, size_t ws_bytes,
                       hipStream_t stream) {
    if (!h || T < 0 || T > h->max_tokens) return EAT_ERR_INVALID_ARG;
    if (!x || !w_router || !mask_out || !k_out || !gate_out) return EAT_ERR_INVALID_ARG;
    if (!aligned(x, 16) || !aligned(w_router, 16) || !aligned(mask_out, 8) || !aligned(k_out, 4) ||
        !aligned(gate_out, 4) || (prob_out && !aligned(prob_out, 4)))
        return EAT_ERR_INVALID_ARG;
    const eat_status_t st = check_accounts(*h, acc);
    if (st != EAT_OK) return st;
    const eat::Workspace w = eat::plan_workspace(*h, T);
    if (T > 0 && (!ws || ws_bytes < w.route_total)) return EAT_ERR_WORKSPACE;
    if (ws && !aligned(ws, 256)) return EAT_ERR_INVALID_ARG;
    if (T == 0) return EAT_OK;
    (void)hipGetLastError();
    const hipError_t e = eat::launch_route(h->p, x, T, w_router, acc, ppl_trend,
                                           reinterpret_cast<float*>(static_cast<char*>(ws) + w.lpart), mask_out,
                                           k_out, gate_out, prob_out, stream);
    return e == hipSuccess ? EAT_OK : EAT_ERR_HIP;
}

}  // extern "C"

namespace eat {

// Argument checks shared by the forward entry points (host only).
eat_status_t check_forward(const eat_ctx* h, const void* x, int32_t T, const float* w_router, const void* w1,
                           const void* w3, const void* w2, const void* ws1, const void* ws3, const void* ws2,
                           const eat_accounts_t& acc, const void* y, const uint64_t* mask_out,
                           const int32_t* expert_load_out) {
    if (!h || T < 0 || T > h->max_tokens) return EAT_ERR_INVALID_ARG;
    const eat_params_t& p = h->p;
    if (!x || !w_router || !w1 || !w3 || !w2 || !y) return EAT_ERR_INVALID_ARG;
    const void* a16[] = {x, w_router, w1, w3, w2, y};
    for (const void* q : a16)
        if (!aligned(q, 16)) return EAT_ERR_INVALID_ARG;
    if (p.d_shared > 0) {
        if (!ws1 || !ws3 || !ws2) return EAT_ERR_INVALID_ARG;
        if (!aligned(ws1, 16) || !aligned(ws3, 16) || !aligned(ws2, 16)) return EAT_ERR_INVALID_ARG;
    } else if (ws1 || ws3 || ws2) {
        return EAT_ERR_INVALID_ARG;
    }
    if ((mask_out && !aligned(mask_out, 8)) || (expert_load_out && !aligned(expert_load_out, 4)))
        return EAT_ERR_INVALID_ARG;
    return check_accounts(*h, acc);
}

// Enqueue one layer forward (arguments already checked, T > 0, workspace
// large enough).  `residual` (bf16 [T][d] or null) is added to y.
hipError_t forward_impl(const eat_ctx& h, const void* x, int32_t T, const float* w_router, const void* w1,
                        const void* w3, const void* w2, const void* ws1, const void* ws3, const void* ws2,
                        eat_accounts_t acc, const int8_t* ppl_trend, const uint16_t* residual, void* y,
                        uint64_t* mask_out, int32_t* expert_load_out, float* prob_out, void* ws,
                        hipStream_t stream, const hipEvent_t* events, int32_t n_events, AccountJob* defer) {
    const eat_params_t& p = h.p;
    const eat::Workspace w = eat::plan_workspace(h, T);
    char* base = static_cast<char*>(ws);
    eat::Buffers b;
    b.lpart = reinterpret_cast<float*>(base + w.lpart);
    b.prob = prob_out ? prob_out : reinterpret_cast<float*>(base + w.prob);
    b.gate = reinterpret_cast<float*>(base + w.gate);
    b.mask = mask_out ? mask_out : reinterpret_cast<uint64_t*>(base + w.mask);
    b.k = reinterpret_cast<int32_t*>(base + w.k);
    b.offsets = reinterpret_cast<int32_t*>(base + w.offsets);
    b.tok_idx = reinterpret_cast<int32_t*>(base + w.tok_idx);
    b.inv = reinterpret_cast<int32_t*>(base + w.inv);
    b.row_expert = reinterpret_cast<int32_t*>(base + w.row_expert);
    b.h = base + w.h;
    b.gu = reinterpret_cast<float*>(base + w.gu);
    b.yp = reinterpret_cast<float*>(base + w.yp);
    b.nrm2 = reinterpret_cast<float*>(base + w.nrm);
    b.hs = base + w.hs;
    b.ys = reinterpret_cast<float*>(base + w.ys);
    b.gus = reinterpret_cast<float*>(base + w.gus);
    b.ysp = reinterpret_cast<float*>(base + w.ysp);
    b.sync = reinterpret_cast<unsigned*>(base + w.sync);
    int32_t* const up_splits_dev = reinterpret_cast<int32_t*>(b.sync);
    int32_t* const down_splits_dev = reinterpret_cast<int32_t*>(b.sync + 1);

    hipError_t e = hipSuccess;
    auto mark = [&](int stage) {
        if (e == hipSuccess && stage < n_events && events[stage]) e = hipEventRecord(events[stage], stream);
    };
    mark(EAT_STAGE_BEGIN);
    if (e == hipSuccess)
        e = eat::launch_route(p, x, T, w_router, acc, ppl_trend, b.lpart, b.mask, b.k, b.gate, b.prob, stream);
    mark(EAT_STAGE_ROUTED);
    if (e == hipSuccess)
        e = eat::launch_permute(p, T, b.mask, b.offsets, b.tok_idx, b.inv, b.row_expert, expert_load_out,
                                stream);
    mark(EAT_STAGE_PERMUTED);
    const bool bf16 = p.expert_dtype == EAT_BF16;
    if (e == hipSuccess) {
        if (bf16)
            e = eat::launch_experts_bf16(p, T, w.rows, static_cast<const uint16_t*>(x),
                                         static_cast<const uint16_t*>(w1), static_cast<const uint16_t*>(w3),
                                         static_cast<const uint16_t*>(w2), b.offsets, b.tok_idx,
                                         static_cast<uint16_t*>(b.h), b.gu, b.yp, b.nrm2, up_splits_dev,
                                         down_splits_dev, stream, [&]() { mark(EAT_STAGE_UP); });
        else
            e = eat::launch_experts_f32(p, T, w.rows, static_cast<const float*>(x),
                                        static_cast<const float*>(w1), static_cast<const float*>(w3),
                                        static_cast<const float*>(w2), b.offsets, b.tok_idx, b.row_expert,
                                        static_cast<float*>(b.h), b.yp, stream, [&]() { mark(EAT_STAGE_UP); });
    }
    mark(EAT_STAGE_DOWN);
    const bool shared = p.d_shared > 0;
    if (e == hipSuccess && shared) {
        if (bf16)
            e = eat::launch_shared_bf16(p, T, static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(ws1),
                                        static_cast<const uint16_t*>(ws3), static_cast<const uint16_t*>(ws2),
                                        static_cast<uint16_t*>(b.hs), b.ys, b.gus, b.ysp, stream);
        else
            e = eat::launch_shared_f32(p, T, static_cast<const float*>(x), static_cast<const float*>(ws1),
                                       static_cast<const float*>(ws3), static_cast<const float*>(ws2),
                                       static_cast<float*>(b.hs), b.ys, stream);
    }
    mark(EAT_STAGE_SHARED);
    // the down projection's slices: chosen on the device when it could take several
    const int32_t* splits_dev = bf16 && w.splits > 1 ? down_splits_dev : nullptr;
    const bool rows16 = bf16 && eat::rows_bf16(p, T);
    if (e == hipSuccess)
        e = eat::launch_combine(p, T, b.mask, b.gate, b.inv, b.yp, shared ? b.ys : nullptr, residual, y, b.nrm2,
                                w.splits, w.rows * p.d_model, splits_dev, rows16, stream);
    mark(EAT_STAGE_COMBINED);
    if (defer) *defer = AccountJob{};
    if (e == hipSuccess && p.mode == EAT_MODE_EAT) {
        if (defer)
            *defer = AccountJob{b.offsets, b.tok_idx, b.prob, b.nrm2, eat::norm_parts(p, T), p.E, p.alpha, acc};
        else
            e = eat::launch_update_accounts(p, b.offsets, b.tok_idx, b.prob, b.nrm2, eat::norm_parts(p, T), acc,
                                            stream);
    }
    mark(EAT_STAGE_END);
    return e;
}

}  // namespace eat

namespace {

using eat::check_forward;
using eat::forward_impl;

// Stacked-layer workspace: the largest layer workspace, then u, r and two
// h rows (bf16 [T][d] each), then the mixing GEMM's fp32 slices.
struct StackPlan {
    size_t layer, u, r, h0, h1, mix, total;
    int splits;
};

StackPlan plan_stack(const eat_stack_layer_t* layers, int32_t n, int32_t T) {
    StackPlan s{};
    auto up = [](size_t v) { return (v + 255) & ~static_cast<size_t>(255); };
    size_t lw = 0;
    for (int32_t l = 0; l < n; ++l) lw = std::max(lw, eat::plan_workspace(*layers[l].layer, T).total);
    const int d = layers[0].layer->p.d_model;
    const size_t row = up(static_cast<size_t>(T) * d * 2);
    s.splits = eat::dense_splits(d, d, T);
    s.layer = 0;
    s.u = up(lw);
    s.r = s.u + row;
    s.h0 = s.r + row;
    s.h1 = s.h0 + row;
    s.mix = s.h1 + row;
    s.total = s.mix + up(static_cast<size_t>(s.splits) * T * d * 4);
    return s;
}

eat_status_t check_stack(const eat_stack_layer_t* layers, int32_t n, int32_t T) {
    if (!layers || n < 1 || n > 1024 || T < 0) return EAT_ERR_INVALID_ARG;
    for (int32_t l = 0; l < n; ++l) {
        const eat_ctx* c = layers[l].layer;
        if (!c || T > c->max_tokens) return EAT_ERR_INVALID_ARG;
        if (c->p.act_dtype != EAT_BF16 || c->p.expert_dtype != EAT_BF16) return EAT_ERR_UNSUPPORTED;
        if (c->p.d_model != layers[0].layer->p.d_model) return EAT_ERR_INVALID_ARG;
        if (!layers[l].mix || !aligned(layers[l].mix, 16)) return EAT_ERR_INVALID_ARG;
    }
    if (!eat::mix_norm_fits(layers[0].layer->p.d_model)) return EAT_ERR_UNSUPPORTED;
    return EAT_OK;
}

}  // namespace

extern "C" {

eat_status_t eat_moe_forward_profiled(eat_handle_t h, const void* x, int32_t T, const float* w_router,
                                      const void* w1, const void* w3, const void* w2, const void* ws1,
                                      const void* ws3, const void* ws2, eat_accounts_t acc,
                                      const int8_t* ppl_trend, void* y, uint64_t* mask_out,
                                      int32_t* expert_load_out, void* ws, size_t ws_bytes, hipStream_t stream,
                                      const hipEvent_t* events, int32_t n_events) {
    if (n_events < 0 || n_events > EAT_NUM_STAGE_EVENTS || (n_events > 0 && !events)) return EAT_ERR_INVALID_ARG;
    const eat_status_t st = check_forward(h, x, T, w_router, w1, w3, w2, ws1, ws3, ws2, acc, y, mask_out,
                                          expert_load_out);
    if (st != EAT_OK) return st;
    const eat::Workspace w = eat::plan_workspace(*h, T);
    if (T > 0 && (!ws || ws_bytes < w.total)) return EAT_ERR_WORKSPACE;
    if (ws && !aligned(ws, 256)) return EAT_ERR_INVALID_ARG;
    if (T == 0) return EAT_OK;
    (void)hipGetLastError();
    const hipError_t e = forward_impl(*h, x, T, w_router, w1, w3, w2, ws1, ws3, ws2, acc, ppl_trend, nullptr, y,
                                      mask_out, expert_load_out, nullptr, ws, stream, events, n_events);
    return e == hipSuccess ? EAT_OK : EAT_ERR_HIP;
}

eat_status_t eat_stack_workspace_size(const eat_stack_layer_t* layers, int32_t n_layers, int32_t T,
                                      size_t* bytes) {
    if (!bytes) return EAT_ERR_INVALID_ARG;
    const eat_status_t st = check_stack(layers, n_layers, T);
    if (st != EAT_OK) return st;
    *bytes = plan_stack(layers, n_layers, T).total;
    return EAT_OK;
}

eat_status_t eat_stack_forward(const eat_stack_layer_t* layers, int32_t n_layers, const void* x, int32_t T,
                               const int8_t* ppl_trend, float rms_eps, void* h_out, uint64_t* masks_out,
                               float* probs_out, void* ws, size_t ws_bytes, hipStream_t stream) {
    eat_status_t st = check_stack(layers, n_layers, T);
    if (st != EAT_OK) return st;
    if (!x || !h_out || !aligned(x, 16) || !aligned(h_out, 16)) return EAT_ERR_INVALID_ARG;
    if ((masks_out && !aligned(masks_out, 8)) || (probs_out && !aligned(probs_out, 4))) return EAT_ERR_INVALID_ARG;
    if (!(rms_eps >= 0.0f) || !std::isfinite(rms_eps)) return EAT_ERR_INVALID_ARG;
    for (int32_t l = 0; l < n_layers; ++l) {
        const eat_stack_layer_t& L = layers[l];
        st = check_forward(L.layer, x, T, L.w_router, L.w1, L.w3, L.w2, L.ws1, L.ws3, L.ws2, L.acc, h_out,
                           masks_out, nullptr);
        if (st != EAT_OK) return st;
    }
    const StackPlan sp = plan_stack(layers, n_layers, T);
    if (T > 0 && (!ws || ws_bytes < sp.total)) return EAT_ERR_WORKSPACE;
    if (ws && !aligned(ws, 256)) return EAT_ERR_INVALID_ARG;
    if (T == 0) return EAT_OK;

    char* base = static_cast<char*>(ws);
    uint16_t* u = reinterpret_cast<uint16_t*>(base + sp.u);
    uint16_t* r = reinterpret_cast<uint16_t*>(base + sp.r);
    uint16_t* hb[2] = {reinterpret_cast<uint16_t*>(base + sp.h0), reinterpret_cast<uint16_t*>(base + sp.h1)};
    float* mix = reinterpret_cast<float*>(base + sp.mix);
    const int d = layers[0].layer->p.d_model;
    const int64_t stride = static_cast<int64_t>(T) * d;

    (void)hipGetLastError();
    size_t prob_off = 0;                      // layer l's probabilities start after T * E_j of the layers before
    size_t mask_off = 0;                      // and its masks after T * mask_words(E_j)
    // u_0 = bf16(RMSNorm(x))
    hipError_t e = eat::launch_mix_norm(nullptr, 0, 0, static_cast<const uint16_t*>(x), T, d, rms_eps, nullptr, u,
                                        nullptr, stream);
    const uint16_t* h = static_cast<const uint16_t*>(x);
    for (int32_t l = 0; l < n_layers && e == hipSuccess; ++l) {
        const eat_stack_layer_t& L = layers[l];
        // r = bf16(h + MoE_l(u)); the layer's account update rides on the
        // RMSNorm launch below (it reads the layer workspace, which the next
        // layer reuses only after that launch)
        eat::AccountJob job{};
        e = forward_impl(*L.layer, u, T, L.w_router, L.w1, L.w3, L.w2, L.ws1, L.ws3, L.ws2, L.acc, ppl_trend, h, r,
                         masks_out ? masks_out + mask_off : nullptr, nullptr,
                         probs_out ? probs_out + prob_off : nullptr, base + sp.layer, stream, nullptr, 0, &job);
        prob_off += static_cast<size_t>(T) * L.layer->p.E;
        mask_off += static_cast<size_t>(T) * eat::mask_words(L.layer->p.E);
        // h' = bf16(r M_l^T); u = bf16(RMSNorm(h')) for the next layer
        if (e == hipSuccess)
            e = eat::launch_dense_bf16(r, T, static_cast<const uint16_t*>(L.mix), d, d, mix, sp.splits, stride,
                                       stream);
        const bool last = l + 1 == n_layers;
        uint16_t* hn = last ? static_cast<uint16_t*>(h_out) : hb[l & 1];
        if (e == hipSuccess)
            e = eat::launch_mix_norm(mix, sp.splits, stride, nullptr, T, d, rms_eps, hn, last ? nullptr : u,
                                     job.experts > 0 ? &job : nullptr, stream);
        h = hn;
    }
    return e == hipSuccess ? EAT_OK : EAT_ERR_HIP;
}

eat_status_t eat_moe_forward(eat_handle_t h, const void* x, int32_t T, const float* w_router,
                             const void* w1, const void* w3, const void* w2, const void* ws1,
                             const void* ws3, const void* ws2, eat_accounts_t acc,
                             const int8_t* ppl_trend, void* y, uint64_t* mask_out,
                             int32_t* expert_load_out, void* ws, size_t ws_bytes, hipStream_t stream) {
    return eat_moe_forward_profiled(h, x, T, w_router, w1, w3, w2, ws1, ws3, ws2, acc, ppl_trend, y, mask_out,
                                    expert_load_out, ws, ws_bytes, stream, nullptr, 0);
}

eat_status_t eat_pack_weights(const void* src, int32_t groups, int32_t M, int32_t K, void* dst,
                              hipStream_t stream) {
    if (!src || !dst || groups < 1 || M < 16 || K < 32 || M % 16 || K % 32) return EAT_ERR_INVALID_ARG;
    if (!aligned(src, 16) || !aligned(dst, 16)) return EAT_ERR_INVALID_ARG;
    const uintptr_t bytes = static_cast<uintptr_t>(groups) * M * K * 2;
    const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
    if (s0 < d0 + bytes && d0 < s0 + bytes) return EAT_ERR_INVALID_ARG;     // overlapping buffers
    (void)hipGetLastError();
    return eat::launch_pack(static_cast<const uint16_t*>(src), groups, M, K, static_cast<uint16_t*>(dst), stream) ==
                   hipSuccess
               ? EAT_OK
               : EAT_ERR_HIP;
}

eat_status_t eat_ppl_workspace_size(int32_t S, int32_t d, int32_t V, size_t* bytes) {
    if (!bytes || S < 0 || S > kMaxTokens || d < 64 || d % 64 || V < 64 || V % 64) return EAT_ERR_INVALID_ARG;
    if (static_cast<int64_t>(d) * V >= (int64_t{1} << 31)) return EAT_ERR_INVALID_ARG;
    *bytes = align256(static_cast<size_t>(eat::ppl_splits(S, d, V)) * S * V * 4) +
             align256(static_cast<size_t>(S) * eat::ppl_chunks(V) * 8);
    return EAT_OK;
}

eat_status_t eat_ppl_reset(int32_t S, double* nll_sum, int32_t* count, double* ppl_prev, hipStream_t stream) {
    if (S < 0 || (S > 0 && (!nll_sum || !count || !ppl_prev))) return EAT_ERR_INVALID_ARG;
    if (!aligned(nll_sum, 8) || !aligned(count, 4) || !aligned(ppl_prev, 8)) return EAT_ERR_INVALID_ARG;
    if (S == 0) return EAT_OK;
    (void)hipGetLastError();
    return eat::launch_ppl_reset(S, nll_sum, count, ppl_prev, stream) == hipSuccess ? EAT_OK : EAT_ERR_HIP;
}

eat_status_t eat_ppl_trend(const void* h, int32_t S, int32_t d, const void* w_vocab, int32_t V,
                           const int32_t* target, double* nll_sum, int32_t* count, double* ppl_prev,
                           int8_t* trend_out, float* nll_out, void* ws, size_t ws_bytes, hipStream_t stream) {
    size_t need = 0;
    const eat_status_t st = eat_ppl_workspace_size(S, d, V, &need);
    if (st != EAT_OK) return st;
    if (S == 0) return EAT_OK;
    if (!h || !w_vocab || !target || !nll_sum || !count || !ppl_prev || !trend_out) return EAT_ERR_INVALID_ARG;
    if (!aligned(h, 16) || !aligned(w_vocab, 16) || !aligned(target, 4) || !aligned(nll_sum, 8) ||
        !aligned(count, 4) || !aligned(ppl_prev, 8) || (nll_out && !aligned(nll_out, 4)))
        return EAT_ERR_INVALID_ARG;
    if (!ws || ws_bytes < need) return EAT_ERR_WORKSPACE;
    if (!aligned(ws, 256)) return EAT_ERR_INVALID_ARG;
    float* z = static_cast<float*>(ws);
    const int splits = eat::ppl_splits(S, d, V);
    const int64_t stride = static_cast<int64_t>(S) * V;
    (void)hipGetLastError();
    hipError_t e = eat::launch_dense_bf16(static_cast<const uint16_t*>(h), S, static_cast<const uint16_t*>(w_vocab),
                                          V, d, z, splits, stride, stream);
    if (e == hipSuccess)
        e = eat::launch_ppl(z, splits, stride, S, V, target, nll_sum, count, ppl_prev, trend_out, nll_out,
                            reinterpret_cast<float2*>(static_cast<char*>(ws) +
                                                      align256(static_cast<size_t>(splits) * S * V * 4)),
                            stream);
    return e == hipSuccess ? EAT_OK : EAT_ERR_HIP;
}

const char* eat_status_string(eat_status_t s) {
    // a C caller may pass any int: read the argument's bits, not the enum
    // (a C++ enum value outside its enumerators' range is undefined)
    int v;
    std::memcpy(&v, &s, sizeof v);
    switch (v) {
        case EAT_OK: return "ok";
        case EAT_ERR_INVALID_ARG: return "invalid argument";
        case EAT_ERR_UNSUPPORTED: return "unsupported shape or dtype";
        case EAT_ERR_WORKSPACE: return "workspace missing or too small";
        case EAT_ERR_HIP: return "HIP runtime error";
        case EAT_ERR_INTERNAL: return "internal error";
        case EAT_ERR_SCRATCH_LIMIT: return "call needs more than the allocation-free entry point's fixed scratch";
    }
    return "unknown status";
}

}  // extern "C"
