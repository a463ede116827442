#!/usr/bin/env python3
"""Benchmark of the EAT MoE-layer forward on one MI355X.

Workload: the Mixtral-8x7B-shaped MoE layer (d_model 4096, 8 SwiGLU experts
of width 14336, bf16 experts, fp32 router and accounts, logits scaled by
1/T with T = 0.5), decode with a batch of 64 tokens per step, hidden states
from a seeded 16-cluster Gaussian mixture (cluster-sticky per sequence,
10% re-draw per step), accounts starting at zero.  A step is one whole
layer forward (route, permute, experts, combine, account update) over one
batch; all inputs are resident in HBM before timing starts.  Steps are
launched eagerly (the host enqueues ahead of the GPU), with HIP events
around the expert kernels of every step.  ``--graph`` also replays one
captured step per step (input copied in, masks copied out inside the timed
region) and reports that as the headline.

Prints one JSON line: EAT tokens/s (``value``), the Top-K (K=2) and Top-P
(p=0.6) baselines on the same inputs, mean activated experts per token,
the experts touched per step, the up/gate kernel's achieved HBM bandwidth
against the MI355X peak (timed per launch with HIP events on the launch
stream), a batch sweep, and the CPU oracle timed on a bounded sample.
An ``eat_cs_share`` object repeats the EAT decode with the other reading of
C_s's scale in S_h (its share C_s,i / sum C_s instead of the raw norm).
A ``stack`` object times the 16-layer workload (16 fine-grained layers,
RMSNorm and a residual mixing matrix between them, decode batch 64) per
routing mode, with every layer's mean activated experts, and EAT with
layer-wise caps (2 in the lower 12 layers, K in the upper 4); a
``ppl_signal`` object times the LM-head perplexity signal (Sec. 3.3) for 64
sequences at the Mixtral head shape.
A ``prefill`` object adds the MFMA-bound side: one prefill call of the
fine-grained layer (4096 tokens, 64 experts of width 1024, K=8), of the
shared-expert layer (8192 tokens, 60 experts of width 1408 + an always-on
expert of width 5632, K=4) and of the Qwen3-30B-A3B-shaped layer (4096
tokens, 128 experts of width 768, K=8), each starting from zero accounts,
with the expert stages' achieved bf16 TFLOP/s against the dense MFMA peak.
A ``wide_experts`` object times decode (batch 64) of that 128-expert layer,
whose selection masks take two 64-bit words per token, and ``decode_layers``
the decode of the fine-grained layer (batch 256, 512 steps) and of the
shared-expert layer (batch 128, 256 steps), each with the whole layer's
algorithmic HBM bandwidth.

    python bench.py [--steps K] [--warmup W] [--batch B] [--gpus 1]
"""
from __future__ import annotations

import argparse
import ctypes as C
import json
import os
import sys
import time
from typing import Optional

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "MoE-layer tokens/s + activated experts/token (EAT vs Top-K); HBM GB/s % peak"
# expert-weight layout every timed layer uses ("packed": eat_pack_weights, set up
# before timing like any weight load; "rows": row-major)
LAYOUT = "packed"


def layout_code() -> int:
    from paper_2609_33614_amd import _lib as L
    return L.EAT_LAYOUT_PACKED if LAYOUT == "packed" else L.EAT_LAYOUT_ROWS


def device_weights(w_host):
    """Host weights -> device tensors in the benchmark's layout."""
    from paper_2609_33614_amd.layer import pack_weights, to_device
    w = to_device(w_host)
    if LAYOUT == "packed":
        packed = pack_weights(w)
        del w
        return packed
    return w
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0          # MI355X dense bf16 MFMA


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class HipEvents:
    """hipEvent_t handles from the HIP runtime, used only for timestamps.

    They are created without the system-scope fence (hipEventDisableSystemFence):
    recording a default event writes back and invalidates the caches, which
    on this part leaves the GPU idle for ~3 us per event (measured: four
    default events per decode step add ~11 us to a 170-280 us step, four
    fence-free ones ~4.5 us).  Nothing here reads device memory through an
    event: every timed region ends with a full device synchronisation."""

    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self):
        self.hip = C.CDLL("libamdhip64.so")
        self.hip.hipEventCreateWithFlags.argtypes = [C.POINTER(C.c_void_p), C.c_uint]
        self.hip.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), C.c_void_p, C.c_void_p]
        self.hip.hipEventDestroy.argtypes = [C.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [C.c_void_p]
        self.owned = []

    def create(self, n: int):
        out = []
        for _ in range(n):
            e = C.c_void_p()
            assert self.hip.hipEventCreateWithFlags(C.byref(e), self.DISABLE_SYSTEM_FENCE) == 0
            out.append(e.value)
        self.owned += out
        return out

    def elapsed_ms(self, a: int, b: int) -> float:
        ms = C.c_float()
        assert self.hip.hipEventSynchronize(b) == 0
        assert self.hip.hipEventElapsedTime(C.byref(ms), a, b) == 0
        return ms.value

    def close(self):
        for e in self.owned:
            self.hip.hipEventDestroy(e)
        self.owned = []


def popcounts(masks: np.ndarray, words: int = 1) -> np.ndarray:
    """Experts selected per token: masks [..., B] (one word per token) or
    [..., B, words]."""
    c = np.bitwise_count(masks.astype(np.uint64)).astype(np.int64)
    return c.sum(axis=-1) if words > 1 else c


def union_sizes(masks: np.ndarray, words: int = 1) -> np.ndarray:
    """Experts touched by any token of each step: masks [steps, B(, words)]."""
    m = masks.astype(np.uint64)
    u = np.bitwise_or.reduce(m, axis=1)
    c = np.bitwise_count(u).astype(np.int64)
    return c.sum(axis=-1) if words > 1 else c


def run_mode(mode, shape, wdev, xs, B, steps, warmup, ev: HipEvents, profile: bool, graph: bool = False,
             cs_mode: int = 0):
    """`steps` timed decode steps after `warmup` untimed ones on scratch
    accounts.  profile: eager launches with HIP events around the expert
    kernels of every step.  graph: one step captured in a HIP graph and
    replayed per step (the step's input copied into the captured buffer and
    its masks copied out, both inside the timed region).  cs_mode: how C_s
    enters S_h (0 raw norm, 1 share of the total)."""
    import torch

    from paper_2609_33614_amd import _lib as L
    from paper_2609_33614_amd.layer import EatLayer, capture

    p = L.eat_params_default(mode=mode, E=shape.E, d_model=shape.d, d_ffn=shape.F, top_k=shape.K,
                             top_p=shape.top_p or 0.6, inv_temperature=shape.inv_temp, d_shared=shape.F_shared,
                             weight_layout=layout_code(), cs_mode=cs_mode)
    lay = EatLayer(p, B, wdev)
    E = shape.E
    W = L.mask_words(E)
    y = torch.empty(B, shape.d, dtype=torch.bfloat16, device="cuda")
    masks = torch.empty((steps, B) if W == 1 else (steps, B, W), dtype=torch.int64, device="cuda")
    scratch = lay.mask_tensor(B)
    # warm-up on a scratch account state, then start from zero accounts
    for s in range(warmup):
        lay.forward(xs[s % xs.shape[0]], y=y, mask_out=scratch)
    x_in = xs[0].clone()
    g = capture(lambda: lay.forward(x_in, y=y, mask_out=scratch)) if graph else None
    lay.reset_accounts()
    torch.cuda.synchronize()

    stage = [None] * L.EAT_NUM_STAGE_EVENTS
    evs = ev.create(4 * steps) if profile else []
    t0, t1 = ev.create(2)
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()
    ev.hip.hipEventRecord.argtypes = [C.c_void_p, C.c_void_p]
    ev.hip.hipEventRecord(t0, stream.cuda_stream)
    for s in range(steps):
        x = xs[warmup + s]
        if g is not None:
            x_in.copy_(x)
            g.replay()
            masks[s].copy_(scratch)
        elif profile:
            stage[L.EAT_STAGE_BEGIN] = evs[4 * s + 3]
            stage[L.EAT_STAGE_PERMUTED] = evs[4 * s]
            stage[L.EAT_STAGE_UP] = evs[4 * s + 1]
            stage[L.EAT_STAGE_DOWN] = evs[4 * s + 2]
            lay.forward(x, y=y, mask_out=masks[s], events=stage)
        else:
            lay.forward(x, y=y, mask_out=masks[s])
    ev.hip.hipEventRecord(t1, stream.cuda_stream)
    torch.cuda.synchronize()
    total_ms = ev.elapsed_ms(t0, t1)
    up_ms = dn_ms = step_ms = None
    if profile:
        up_ms = np.array([ev.elapsed_ms(evs[4 * s], evs[4 * s + 1]) for s in range(steps)])
        dn_ms = np.array([ev.elapsed_ms(evs[4 * s + 1], evs[4 * s + 2]) for s in range(steps)])
        # a step runs from its first event to the next step's (the last one to the end event)
        begins = [evs[4 * s + 3] for s in range(steps)] + [t1]
        step_ms = np.array([ev.elapsed_ms(begins[s], begins[s + 1]) for s in range(steps)])
    m = masks.cpu().numpy().astype(np.int64).view(np.uint64)
    k = popcounts(m, W)
    U = union_sizes(m, W)
    acc = lay.accounts_host()
    del g
    lay.close()
    return dict(total_ms=total_ms, up_ms=up_ms, dn_ms=dn_ms, step_ms=step_ms, k=k, U=U, E=E, accounts=acc,
                masks=m, words=W)


def routing_stats(res, K: int) -> dict:
    """Routing statistics of a decode run: how many tokens activated each
    number of experts, the tokens above the cap K (Eq. 6 keeps every exact
    tie at the K-th value, so EAT may exceed K only on exact ties), each
    expert's share of the (token, expert) assignments, and the experts
    touched per step."""
    k, m, W, E = res["k"], res["masks"], res["words"], res["E"]
    hist = np.bincount(k.ravel())
    load = np.zeros(E, dtype=np.int64)
    for e in range(E):
        word = m[..., e // 64] if W > 1 else m
        load[e] = int(((word >> np.uint64(e % 64)) & np.uint64(1)).sum())
    U = res["U"]
    return {"k_histogram": {str(i): int(c) for i, c in enumerate(hist) if c},
            "tokens_above_cap": int((k > K).sum()),
            "expert_load_share": [round(float(v), 4) for v in load / max(1, load.sum())],
            "experts_touched_min_mean_max": [int(U.min()), round(float(U.mean()), 3), int(U.max())]}


def trajectory(res, B: int, first: int = 20, settle: int = 64) -> dict:
    """Per-step view of a decode run from zero accounts: the experts touched
    at every step, and tokens/s over the first `first` steps (the history
    still building up) against the steps after `settle`."""
    sm, U = res["step_ms"], res["U"]
    n = len(sm)
    out = {"steps": n, "experts_touched_per_step": [int(u) for u in U]}
    f = min(first, n)
    out[f"first_{f}_steps"] = {"tokens_per_s": round(B * f / (sm[:f].sum() / 1e3), 1),
                               "ms_per_step": round(float(sm[:f].mean()), 4),
                               "mean_experts_touched": round(float(U[:f].mean()), 3)}
    if n > settle:
        out[f"steps_{settle}_to_{n}"] = {"tokens_per_s": round(B * (n - settle) / (sm[settle:].sum() / 1e3), 1),
                                          "ms_per_step": round(float(sm[settle:].mean()), 4),
                                          "mean_experts_touched": round(float(U[settle:].mean()), 3)}
    return out


def run_prefill(shape_name: str, reps: int, ev: HipEvents, modes=("eat", "topk")):
    """One prefill call of a layer (its prompt tokens, zero accounts) timed
    per stage with HIP events, `reps` times after 2 untimed calls; returns
    per-mode tokens/s, activated experts and the expert stages' TFLOP/s."""
    import torch

    from paper_2609_33614_amd import _lib as L
    from paper_2609_33614_amd.layer import EatLayer, to_device
    from workload import SHAPES, make_layer_weights, make_prefill

    shape = SHAPES[shape_name]
    T = shape.prefill_tokens
    wdev = device_weights(make_layer_weights(shape))
    x = torch.from_numpy(make_prefill(shape)).view(torch.bfloat16).cuda()
    y = torch.empty(T, shape.d, dtype=torch.bfloat16, device="cuda")
    W = L.mask_words(shape.E)
    mask = torch.empty((T,) if W == 1 else (T, W), dtype=torch.int64, device="cuda")
    d, F, Fs, E = shape.d, shape.F, shape.F_shared, shape.E
    out = {"workload": f"{shape_name} layer prefill", "tokens": T, "d_model": d, "experts": E, "d_ffn": F,
           "d_shared": Fs, "top_k": shape.K}
    for mode in modes:
        p = L.eat_params_default(mode=L.MODES[mode], E=E, d_model=d, d_ffn=F, top_k=shape.K,
                                 top_p=shape.top_p or 0.6, inv_temperature=shape.inv_temp, d_shared=Fs,
                                 weight_layout=layout_code())
        lay = EatLayer(p, T, wdev)
        stage = ev.create(L.EAT_NUM_STAGE_EVENTS)
        tot, up, dn, sh = [], [], [], []
        for it in range(2 + reps):
            lay.reset_accounts()
            lay.forward(x, y=y, mask_out=mask, events=stage)
            torch.cuda.synchronize()
            if it >= 2:
                tot.append(ev.elapsed_ms(stage[L.EAT_STAGE_BEGIN], stage[L.EAT_STAGE_END]))
                up.append(ev.elapsed_ms(stage[L.EAT_STAGE_PERMUTED], stage[L.EAT_STAGE_UP]))
                dn.append(ev.elapsed_ms(stage[L.EAT_STAGE_UP], stage[L.EAT_STAGE_DOWN]))
                sh.append(ev.elapsed_ms(stage[L.EAT_STAGE_DOWN], stage[L.EAT_STAGE_SHARED]))
        lay.close()
        sk = float(popcounts(mask.cpu().numpy().astype(np.int64).view(np.uint64)[None], W).sum())
        t_ms, up_ms, dn_ms, sh_ms = (float(np.median(v)) for v in (tot, up, dn, sh))
        fl_up, fl_dn = 4.0 * d * F * sk, 2.0 * d * F * sk
        fl_sh = 6.0 * d * Fs * T
        fl_all = 2.0 * T * d * E + fl_up + fl_dn + fl_sh
        tf = lambda fl, ms: fl / (ms * 1e-3) / 1e12
        r = {"tokens_per_s": round(T / (t_ms * 1e-3), 1), "ms": round(t_ms, 4),
             "mean_activated_experts": round(sk / T, 4),
             "up_gate": {"us": round(up_ms * 1e3, 1), "tflops": round(tf(fl_up, up_ms), 1),
                         "frac": round(tf(fl_up, up_ms) / BF16_PEAK_TFLOPS, 4)},
             "down": {"us": round(dn_ms * 1e3, 1), "tflops": round(tf(fl_dn, dn_ms), 1),
                      "frac": round(tf(fl_dn, dn_ms) / BF16_PEAK_TFLOPS, 4)},
             "layer_tflops": round(tf(fl_all, t_ms), 1)}
        if Fs:
            r["shared"] = {"us": round(sh_ms * 1e3, 1), "tflops": round(tf(fl_sh, sh_ms), 1),
                           "frac": round(tf(fl_sh, sh_ms) / BF16_PEAK_TFLOPS, 4)}
        out[mode] = r
    del wdev
    torch.cuda.empty_cache()
    return out


def run_decode(shape_name: str, steps: Optional[int], warmup: int, ev: HipEvents, modes=("eat", "topk", "topp")):
    """Decode steps of one more layer shape (its own decode batch, zero
    accounts after warm-up; `steps` timed steps, or the layer's own count
    when None) per routing mode: tokens/s, activated experts, experts
    touched, the routed expert kernels' achieved HBM bandwidth on their
    algorithmic bytes, and the whole layer's (experts touched, the always-on
    expert, router, token rows in and out) against the step time."""
    import torch

    from paper_2609_33614_amd import _lib as L
    from paper_2609_33614_amd.layer import to_device
    from workload import SHAPES, HiddenStream, make_layer_weights

    shape = SHAPES[shape_name]
    B = shape.decode_batches[0]
    steps = shape.decode_steps if steps is None else steps
    wdev = device_weights(make_layer_weights(shape))
    xs = torch.from_numpy(HiddenStream(shape, B).steps(warmup + steps)).view(torch.bfloat16).cuda()
    out = {"workload": f"{shape_name} layer decode", "batch": B, "d_model": shape.d, "experts": shape.E,
           "d_ffn": shape.F, "d_shared": shape.F_shared, "top_k": shape.K, "mask_words": L.mask_words(shape.E),
           "steps": steps}
    for name in modes:
        r = run_mode(L.MODES[name], shape, wdev, xs, B, steps, warmup, ev, profile=True)
        up_b = sum(traffic_up(shape, B, r["k"][s], r["U"][s]) for s in range(steps))
        dn_b = sum(traffic_down(shape, r["k"][s], r["U"][s]) for s in range(steps))
        up_gbs = up_b / (r["up_ms"].sum() / 1e3) / 1e9
        dn_gbs = dn_b / (r["dn_ms"].sum() / 1e3) / 1e9
        layer_b = (r["U"].sum() * 3.0 * shape.d * shape.F * 2 +
                   steps * (3.0 * shape.d * shape.F_shared * 2 + shape.E * shape.d * 4 + 2.0 * B * shape.d * 2))
        out[name] = {"tokens_per_s": round(B * steps / (r["total_ms"] / 1e3), 1),
                     "ms_per_step": round(r["total_ms"] / steps, 4),
                     "mean_activated_experts": round(float(r["k"].mean()), 4),
                     "mean_experts_touched_per_step": round(float(r["U"].mean()), 3),
                     "up_gate_us_per_launch": round(float(r["up_ms"].mean() * 1e3), 2),
                     "up_gate_hbm_frac": round(up_gbs / HBM_PEAK_GBS, 4),
                     "down_us_per_launch": round(float(r["dn_ms"].mean() * 1e3), 2),
                     "down_hbm_frac": round(dn_gbs / HBM_PEAK_GBS, 4),
                     "layer_hbm_frac": round(layer_b / (r["total_ms"] / 1e3) / 1e9 / HBM_PEAK_GBS, 4)}
        log(f"{shape_name} decode {name}: {out[name]['tokens_per_s']} tok/s")
    del wdev, xs
    torch.cuda.empty_cache()
    return out


def run_stack(steps: int, warmup: int, ev: HipEvents, modes=("eat", "topk", "topp", "eat_layerwise")):
    """The 16-layer workload: decode batch 64 through 16 stacked fine-grained
    layers (own accounts each, RMSNorm + residual mixing between layers),
    `steps` timed steps per mode after `warmup` untimed ones on scratch
    accounts (then reset).  Returns per-mode tokens/s, per-layer mean
    activated experts and experts touched, and the step's algorithmic HBM
    bandwidth (every layer's router, the experts its tokens touch, its mixing
    matrix)."""
    import torch

    from paper_2609_33614_amd import _lib as L
    from paper_2609_33614_amd.layer import EatStack, layerwise_caps, to_device
    from workload import SHAPES, HiddenStream, make_layer_weights, make_mixing

    shape = SHAPES["stack16"]
    nl, B, d, E, F = shape.layers, shape.decode_batches[0], shape.d, shape.E, shape.F
    t = time.time()
    wdev, mdev = [], []
    for l in range(nl):
        wdev.append(device_weights(make_layer_weights(shape, layer=l)))
        mdev.append(torch.from_numpy(make_mixing(shape, l)).view(torch.bfloat16).cuda())
    log(f"stack weights ready in {time.time() - t:.1f} s ({nl} layers)")
    xs = torch.from_numpy(HiddenStream(shape, B).steps(warmup + steps)).view(torch.bfloat16).cuda()
    out = {"workload": f"{nl}-layer stack decode (RMSNorm + residual mixing between layers)", "layers": nl,
           "batch": B, "d_model": d, "experts": E, "d_ffn": F, "top_k": shape.K, "steps": steps}
    for mode in modes:
        # eat_layerwise: layer-wise sparsity, EAT capped at 2 in the lower 12
        # layers and at the model's K in the upper 4
        caps = layerwise_caps(nl, 12, 2, shape.K) if mode == "eat_layerwise" else [shape.K] * nl
        rmode = "eat" if mode == "eat_layerwise" else mode
        params = [L.eat_params_default(mode=L.MODES[rmode], E=E, d_model=d, d_ffn=F, top_k=caps[l],
                                       top_p=shape.top_p, inv_temperature=shape.inv_temp,
                                       weight_layout=layout_code()) for l in range(nl)]
        st = EatStack(params, B, wdev, mdev)
        h = torch.empty(B, d, dtype=torch.bfloat16, device="cuda")
        masks = torch.empty(steps, nl, B, dtype=torch.int64, device="cuda")
        scratch = torch.empty(nl, B, dtype=torch.int64, device="cuda")
        for s_ in range(warmup):
            st.forward(xs[s_], h_out=h, masks_out=scratch)
        st.reset_accounts()
        t0, t1 = ev.create(2)
        stream = torch.cuda.current_stream().cuda_stream
        torch.cuda.synchronize()
        ev.hip.hipEventRecord.argtypes = [C.c_void_p, C.c_void_p]
        ev.hip.hipEventRecord(t0, stream)
        for s_ in range(steps):
            st.forward(xs[warmup + s_], h_out=h, masks_out=masks[s_])
        ev.hip.hipEventRecord(t1, stream)
        torch.cuda.synchronize()
        ms = ev.elapsed_ms(t0, t1)
        m = masks.cpu().numpy().astype(np.int64).view(np.uint64)                # [steps, layers, B]
        k = np.stack([popcounts(m[:, l, :]) for l in range(nl)])                # [layers, steps, B]
        U = np.stack([union_sizes(m[:, l, :]) for l in range(nl)])              # [layers, steps]
        st.close()
        bytes_step = (U.sum(axis=0) * 3.0 * d * F * 2 + nl * (E * d * 4 + d * d * 2 + B * d * 2 * 4)).mean()
        out[mode] = {"tokens_per_s": round(B * steps / (ms / 1e3), 1), "ms_per_step": round(ms / steps, 4),
                     "mean_activated_experts": round(float(k.mean()), 4),
                     "per_layer_mean_activated_experts": [round(float(v), 3) for v in k.mean(axis=(1, 2))],
                     "per_layer_experts_touched": [round(float(v), 2) for v in U.mean(axis=1)],
                     "hbm_gbs": round(bytes_step / (ms / steps / 1e3) / 1e9, 1),
                     "hbm_frac": round(bytes_step / (ms / steps / 1e3) / 1e9 / HBM_PEAK_GBS, 4)}
        log(f"stack {mode}: {out[mode]['tokens_per_s']} tok/s, {out[mode]['ms_per_step']} ms/step")
    del wdev, mdev
    torch.cuda.empty_cache()
    return out


def run_ppl(ev: HipEvents, S: int = 64, d: int = 4096, V: int = 32000, reps: int = 50):
    """The perplexity signal (LM-head NLL, running perplexity, trend) for S
    sequences at the Mixtral head shape: microseconds per call and the
    achieved bandwidth on its algorithmic bytes (W_V, the hidden rows, the
    fp32 logits written and read once, the state)."""
    import torch

    from paper_2609_33614_amd.layer import PplSignal
    from workload import SHAPES, HiddenStream, make_targets, make_vocab_head

    w = torch.from_numpy(make_vocab_head(d, V, seed=1)).view(torch.bfloat16).cuda()
    h = torch.from_numpy(HiddenStream(SHAPES["mixtral"], S).next()).view(torch.bfloat16).cuda()
    y = torch.from_numpy(make_targets(S, V, seed=2)).cuda()
    sig = PplSignal(S, w)
    sig.reset()
    for _ in range(5):
        sig.step(h, y)
    t0, t1 = ev.create(2)
    stream = torch.cuda.current_stream().cuda_stream
    torch.cuda.synchronize()
    ev.hip.hipEventRecord.argtypes = [C.c_void_p, C.c_void_p]
    ev.hip.hipEventRecord(t0, stream)
    for _ in range(reps):
        sig.step(h, y)
    ev.hip.hipEventRecord(t1, stream)
    torch.cuda.synchronize()
    us = ev.elapsed_ms(t0, t1) / reps * 1e3
    nbytes = V * d * 2 + S * d * 2 + 2 * S * V * 4 + S * 21
    return {"workload": "LM-head perplexity signal", "sequences": S, "d_model": d, "vocab": V,
            "us_per_call": round(us, 2), "hbm_gbs": round(nbytes / (us * 1e-6) / 1e9, 1),
            "hbm_frac": round(nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}


def traffic_up(shape, B, k_row, U):
    """Algorithmic HBM bytes of one up/gate launch: W1 and W3 rows of every
    expert in the step's union, the B token rows read, the H rows written."""
    d, F = shape.d, shape.F
    return U * 2 * F * d * 2 + B * d * 2 + k_row.sum() * F * 2


def traffic_down(shape, k_row, U):
    """Algorithmic HBM bytes of one down launch: W2 of every expert in the
    union, the H rows read, one fp32 output row per (token, expert)."""
    d, F = shape.d, shape.F
    return U * d * F * 2 + k_row.sum() * F * 2 + k_row.sum() * d * 4


def measured_traffic(prefix: str, batch: int, steps: int, warmup: int):
    """HBM bytes per launch of the dominant kernel from a committed counter
    summary profiles/<prefix>*.traffic.txt taken on a run with this batch and
    these timed and warm-up steps (the experts a step touches, and so the
    bytes per launch, depend on how far the account history has built up),
    or None when there is none or it was measured on a different version of
    the expert kernel source."""
    import glob
    import hashlib
    sha = hashlib.sha1(open(os.path.join(ROOT, "paper_2609_33614_amd", "csrc", "expert.hip"), "rb").read()).hexdigest()
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", prefix + "*.traffic.txt"))):
        kv = dict(line.split(": ", 1) for line in open(path).read().splitlines() if ": " in line)
        if (kv.get("source_sha1") == sha and kv.get("batch") == str(batch) and kv.get("steps") == str(steps)
                and kv.get("warmup") == str(warmup)):
            return float(kv["traffic_bytes_per_launch"])
    return None


def _oracle_rate(shape, w_host, xs_host, B, max_seconds: float):
    """Steps of the oracle (unchanged) on the same EAT decode from zero
    accounts until `max_seconds` have passed: (steps, seconds)."""
    import oracle as O
    prm = O.Params(mode=O.MODE_EAT, K=shape.K, inv_temp=shape.inv_temp)
    acc = O.zero_accounts(shape.E)
    t = time.time()
    n = 0
    while True:
        out = O.moe_step(xs_host[n], w_host, acc, None, prm)
        acc = out.acc
        n += 1
        if time.time() - t >= max_seconds or n >= xs_host.shape[0]:
            break
    return n, time.time() - t


def cpu_baseline(shape, w_host, xs_host, B, max_seconds: float, single_seconds: float):
    """The oracle, unchanged, on the first steps of the same EAT workload:
    with the BLAS threads the host gives it, and again with one thread."""
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        blas = [i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"]
        cores = int(max(blas)) if blas else 1
    except Exception:
        threadpool_limits, cores = None, 1
    n, dt = _oracle_rate(shape, w_host, xs_host, B, max_seconds)
    out = {"value": round(n * B / dt, 3), "unit": "tokens/s", "cores": cores, "kind": "oracle",
           "sample": f"{n} EAT decode step(s) of B={B} on the same layer and inputs "
                     f"({n * B} tokens, {dt:.1f} s; numpy fp64, BLAS threads={cores})"}
    if threadpool_limits is not None and single_seconds > 0:
        with threadpool_limits(limits=1, user_api="blas"):
            n1, dt1 = _oracle_rate(shape, w_host, xs_host, B, single_seconds)
        out["single_thread"] = {"value": round(n1 * B / dt1, 3), "unit": "tokens/s", "cores": 1,
                                "sample": f"{n1} step(s), {n1 * B} tokens, {dt1:.1f} s, BLAS threads=1"}
    return out


def oracle_workloads(decode_seconds: float):
    """The oracle (unchanged) on the fine-grained and shared-expert layers:
    EAT decode steps from zero accounts (at least one, until
    `decode_seconds` have passed) at the layer's decode batch, then one
    prefill call at its prefill size, each on the host's BLAS threads."""
    import oracle as O
    from workload import SHAPES, HiddenStream, make_layer_weights

    out = []
    for name, T in (("finegrained", 4096), ("shared", 8192)):
        shape = SHAPES[name]
        B = shape.decode_batches[0]
        w = make_layer_weights(shape)
        prm = O.Params(mode=O.MODE_EAT, K=shape.K, inv_temp=shape.inv_temp)
        xs = HiddenStream(shape, B).steps(64)
        acc = O.zero_accounts(shape.E)
        t = time.time()
        n = 0
        while n < xs.shape[0]:
            acc = O.moe_step(xs[n], w, acc, None, prm).acc
            n += 1
            if time.time() - t >= decode_seconds:
                break
        dt = time.time() - t
        xp = HiddenStream(shape, T).steps(1)[0]
        t = time.time()
        O.moe_step(xp, w, O.zero_accounts(shape.E), None, prm)
        dp = time.time() - t
        out.append({"workload": f"{name} layer", "decode": {"value": round(n * B / dt, 3), "unit": "tokens/s",
                                                           "sample": f"{n} EAT step(s) of B={B}, {dt:.1f} s"},
                    "prefill": {"value": round(T / dp, 3), "unit": "tokens/s",
                                "sample": f"one EAT call of {T} tokens, {dp:.1f} s"}})
        del w
    return out


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=256)
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--batch", type=int, default=64)
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--cpu-single-seconds", type=float, default=10.0,
                    help="seconds of the one-BLAS-thread oracle timing (0 = skip)")
    ap.add_argument("--cpu-workload-seconds", type=float, default=3.0,
                    help="seconds of oracle decode steps on each of the fine-grained and shared-expert layers, "
                         "each followed by one prefill call (0 = skip both)")
    ap.add_argument("--modes", default="eat,topk,topp", help="routing modes to time (eat first)")
    ap.add_argument("--no-prefill", action="store_true", help="skip the prefill (MFMA-bound) measurement")
    ap.add_argument("--prefill-reps", type=int, default=10)
    ap.add_argument("--graph", action="store_true",
                    help="also time the decode steps as HIP graph replays and report those as the headline")
    ap.add_argument("--no-stack", action="store_true", help="skip the 16-layer stack measurement")
    ap.add_argument("--layout", choices=("packed", "rows"), default="packed",
                    help="expert-weight layout of every timed layer (default: packed)")
    ap.add_argument("--no-wide-experts", action="store_true",
                    help="skip the decode of the 128-expert (Qwen3-30B-A3B-shaped) layer")
    ap.add_argument("--no-trajectory", action="store_true",
                    help="skip the 256-step EAT trajectory object (taken from the timed run when --steps >= 256)")
    ap.add_argument("--no-share", action="store_true",
                    help="skip the EAT decode under the C_s-share reading (cs_mode 1)")
    ap.add_argument("--no-decode-layers", action="store_true",
                    help="skip the decode of the fine-grained (B=256) and shared-expert (B=128) layers")
    ap.add_argument("--stack-steps", type=int, default=1024)
    ap.add_argument("--only-stack", action="store_true", help="time only the 16-layer stack and print its JSON")
    ap.add_argument("--only-decode-layer", default="", metavar="LAYER",
                    help="time only one decode_layers workload (finegrained or shared) and print its JSON")
    ap.add_argument("--only-prefill", default="", metavar="LAYER",
                    help="time only the prefill of LAYER (finegrained or shared) in --modes and print "
                         "its JSON object (for kernel traces of the MFMA-bound path)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="also run 4 plain device copies of MIB MiB (a known-size kernel for "
                         "calibrating HBM byte counters)")
    args = ap.parse_args(argv)
    global LAYOUT
    LAYOUT = args.layout
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the EAT layer path here is a single-GPU build "
              f"(asked for --gpus {args.gpus}, WORLD_SIZE {world}).", file=sys.stderr)
        return 2

    import torch

    from paper_2609_33614_amd import _lib as L
    from paper_2609_33614_amd.layer import to_device
    from workload import SHAPES, HiddenStream, make_layer_weights

    L.load()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.only_stack:
        ev = HipEvents()
        res = run_stack(args.stack_steps, 16, ev, modes=[m for m in args.modes.split(",") if m])
        ev.close()
        print(json.dumps({"stack": res}), flush=True)
        return 0
    if args.only_decode_layer:
        ev = HipEvents()
        res = run_decode(args.only_decode_layer, None, args.warmup, ev,
                         modes=[m for m in args.modes.split(",") if m])
        ev.close()
        print(json.dumps({"decode_layers": [res]}), flush=True)
        return 0
    if args.only_prefill:
        ev = HipEvents()
        res = run_prefill(args.only_prefill, args.prefill_reps, ev, modes=[m for m in args.modes.split(",") if m])
        ev.close()
        print(json.dumps({"prefill": [res]}), flush=True)
        return 0
    shape = SHAPES["mixtral"]
    B, K, W = args.batch, args.steps, args.warmup
    log(f"generating weights d={shape.d} E={shape.E} F={shape.F}")
    t = time.time()
    w_host = make_layer_weights(shape)
    wdev = device_weights(w_host)
    TRAJ = 256                        # steps of the from-zero EAT trajectory object
    log(f"weights ready in {time.time() - t:.1f} s; generating {W + max(K, TRAJ)} steps of B={B}")
    xs_host = HiddenStream(shape, B).steps(W + max(K, TRAJ))
    xs = torch.from_numpy(xs_host).view(torch.bfloat16).cuda()
    ev = HipEvents()

    if args.calibrate_copy:
        n = args.calibrate_copy * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(4):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log(f"copy calibration: 4 x {args.calibrate_copy} MiB read + written")

    results, graphed = {}, {}
    modes = [m for m in args.modes.split(",") if m]
    assert modes and modes[0] == "eat", "the headline mode (eat) is timed first"
    for name in modes:
        log(f"timing {name}: {K} steps (+{W} warm-up), eager with kernel events")
        results[name] = run_mode(L.MODES[name], shape, wdev, xs, B, K, W, ev, profile=True)
        if args.graph:
            log(f"timing {name}: {K} steps (+{W} warm-up), HIP graph replay")
            graphed[name] = run_mode(L.MODES[name], shape, wdev, xs, B, K, W, ev, profile=False, graph=True)
    # the same EAT decode over 256 steps: how the step time follows the
    # experts touched as the account history builds up
    traj = results["eat"] if K >= TRAJ else None
    if traj is None and not args.no_trajectory:
        log(f"timing eat: {TRAJ} steps (+{W} warm-up) for the per-step trajectory")
        traj = run_mode(L.MODES["eat"], shape, wdev, xs, B, TRAJ, W, ev, profile=True)
    share = None
    if not args.no_share:
        log(f"timing eat with the C_s-share reading: {K} steps (+{W} warm-up)")
        share = run_mode(L.MODES["eat"], shape, wdev, xs, B, K, W, ev, profile=True, cs_mode=1)
    r = results["eat"]
    head = graphed.get("eat", r)
    ms_step = head["total_ms"] / K
    value = B * K / (head["total_ms"] / 1e3)

    up_bytes = np.array([traffic_up(shape, B, r["k"][s], r["U"][s]) for s in range(K)], dtype=np.float64)
    dn_bytes = np.array([traffic_down(shape, r["k"][s], r["U"][s]) for s in range(K)], dtype=np.float64)
    up_gbs = up_bytes.sum() / (r["up_ms"].sum() / 1e3) / 1e9
    dn_gbs = dn_bytes.sum() / (r["dn_ms"].sum() / 1e3) / 1e9

    def summary(res, gres):
        best = gres if gres is not None else res
        return {"tokens_per_s": round(B * K / (best["total_ms"] / 1e3), 1),
                "ms_per_step": round(best["total_ms"] / K, 4),
                "eager_tokens_per_s": round(B * K / (res["total_ms"] / 1e3), 1),
                "mean_activated_experts": round(float(res["k"].mean()), 4),
                "mean_experts_touched_per_step": round(float(res["U"].mean()), 3),
                "up_gate_us_per_launch": round(float(res["up_ms"].mean() * 1e3), 2),
                "down_us_per_launch": round(float(res["dn_ms"].mean() * 1e3), 2),
                "routing": routing_stats(res, shape.K)}

    sweep = []
    if not args.no_sweep:
        for b in (1, 8, 32):
            xb = torch.from_numpy(HiddenStream(shape, b).steps(W + K)).view(torch.bfloat16).cuda()
            row = {"batch": b}
            for name in ("eat", "topk"):
                log(f"sweep B={b} {name}")
                rr = run_mode(L.MODES[name], shape, wdev, xb, b, K, W, ev, profile=False, graph=args.graph)
                row[name] = {"tokens_per_s": round(b * K / (rr["total_ms"] / 1e3), 1),
                             "ms_per_step": round(rr["total_ms"] / K, 4),
                             "mean_activated_experts": round(float(rr["k"].mean()), 4),
                             "mean_experts_touched_per_step": round(float(rr["U"].mean()), 3)}
            sweep.append(row)
            del xb
    prefill = []
    if not args.no_prefill:
        del wdev
        torch.cuda.empty_cache()
        for name in ("finegrained", "shared", "qwen3"):
            log(f"prefill {name}: {args.prefill_reps} timed calls per mode")
            prefill.append(run_prefill(name, args.prefill_reps, ev))
    wide_e = None
    if not args.no_wide_experts:
        if "wdev" in locals():
            del wdev
            torch.cuda.empty_cache()
        log("qwen3-shaped layer decode (128 experts)")
        wide_e = run_decode("qwen3", K, W, ev)
    decode_layers = []
    if not args.no_decode_layers:
        if "wdev" in locals():
            del wdev
            torch.cuda.empty_cache()
        for name, dmodes in (("finegrained", ("eat", "topk", "topp")), ("shared", ("eat", "topk"))):
            log(f"{name}-layer decode ({SHAPES[name].decode_steps} steps of B={SHAPES[name].decode_batches[0]})")
            decode_layers.append(run_decode(name, None, W, ev, modes=dmodes))
    log("perplexity signal")
    ppl = run_ppl(ev)
    stack = None
    if not args.no_stack:
        if "wdev" in locals():
            del wdev
            torch.cuda.empty_cache()
        stack = run_stack(args.stack_steps, 16, ev)
    ev.close()

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        cpu = cpu_baseline(shape, w_host, xs_host[W:], B, args.cpu_seconds, args.cpu_single_seconds)
        if args.cpu_workload_seconds > 0:
            log("timing the CPU oracle on the fine-grained and shared-expert layers")
            del w_host
            cpu["other_workloads"] = oracle_workloads(args.cpu_workload_seconds)

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded Gaussian-mixture hidden states, random-init weights)",
        "config": {"workload": "Mixtral-shaped MoE layer decode, EAT routing",
                   "d_model": shape.d, "experts": shape.E, "d_ffn": shape.F, "top_k": shape.K,
                   "batch": B, "logit_scale": shape.inv_temp, "router": "fp32", "experts_dtype": "bf16",
                   "launch": "HIP graph replay per step" if args.graph else "eager",
                   "weight_layout": LAYOUT},
        "roofline": {"bound": "hbm", "kernel": "expert up/gate (stream_kernel<gated>)",
                     "achieved": round(up_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(up_gbs / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic("up_gate_mixtral_decode_b64_eat", B, K, W),
                     "down_achieved": round(dn_gbs, 1),
                     "bytes_per_launch": round(float(up_bytes.mean()), 0),
                     "us_per_launch": round(float(r["up_ms"].mean() * 1e3), 2)},
        "cpu_baseline": cpu,
        "modes": {name: summary(res, graphed.get(name)) for name, res in results.items()},
        "eat_cs_share": dict(summary(share, None), reading="C_s enters S_h as C_s,i / sum C_s (cs_mode 1)")
        if share is not None else None,
        "eat_trajectory": trajectory(traj, B) if traj is not None else None,
        "sweep": sweep,
        "prefill": prefill,
        "stack": stack,
        "ppl_signal": ppl,
        "wide_experts": wide_e,
        "decode_layers": decode_layers,
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
