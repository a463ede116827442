"""GPU parity of the stacked-layer step (eat_stack_forward) against the
oracle's stack_step: per-layer selection masks and router probabilities,
the final hidden rows and every layer's accounts.

The oracle rounds the experts' hidden activation to bf16 here as the GPU
stores it (reading R27, ``round_h``): left exact, that rounding alone
(~5e-3 of a layer's output) would reach every later router.  What remains
is that each side rounds r, h and u to bf16 from its own value (fp32 on the
GPU, fp64 in the oracle), so an element near a rounding boundary can differ
by one bf16 step and reach the next router.  The borderline band of a token
at a layer is therefore 4x its own largest |p_gpu - p_oracle| there (never
below the single-layer band, and that difference itself must stay below the
case's ceiling); tokens within it, and everything they feed in later
layers, are excluded from the bit-exact mask comparison and counted.  From
the second EAT step on, the two sides' account states differ a little too
(P_total by the summed |dp|, C_s by the output norms); with N equal, Eq. 1
bounds the history score's difference by w2 |dP_total| / N + w3 |dC_s|, and
beta times that joins every token's band at that layer.

Most tokens never meet such a boundary: the median |p_gpu - p_oracle| over
the tokens of every layer must stay at the single-layer level.

With W2 = 0 the experts add exactly zero on both sides, so the stack
reduces to RMSNorm, routing, residual and mixing.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_33614_amd import _lib as L
from paper_2609_33614_amd.layer import EatStack, to_device
from workload import SHAPES, HiddenStream, make_layer_weights, make_mixing

from tests import parity as PT

pytestmark = pytest.mark.gpu

# |p_gpu - p_oracle| on tokens whose path has not diverged: one bf16 step
# (2**-8 relative) in an element of r or h reaches the next router as ~2.5e-4
# relative in u, and such steps compound over the layers; a wrong kernel
# shows up as ~1e-1
DP_CEIL = 2e-3
DP_MEDIAN = 1e-6      # median of that over the tokens of a layer
TOL_H = 2e-2          # per-token max|dh| / max|h| after the last layer
# share of tokens a step may exclude: with 64 experts a band of a few 1e-4
# around tau_final holds some expert of many tokens
MAX_TAINTED = {16: 0.25, 64: 0.5}


def _build(mode, n_layers, d, E, F, B, seed=None, zero_w2=False, caps=None):
    shape = SHAPES["stack16"]
    caps = caps or [shape.K] * n_layers
    w_host = [make_layer_weights(shape, seed=seed, layer=l, E=E, d=d, F=F) for l in range(n_layers)]
    if zero_w2:
        for w in w_host:
            w["w2"] = np.zeros_like(w["w2"])
    mixes = [make_mixing(shape, l, seed=seed, d=d) for l in range(n_layers)]
    params = [L.eat_params_default(mode=L.MODES[mode], E=E, d_model=d, d_ffn=F, top_k=caps[l], top_p=shape.top_p,
                                   inv_temperature=shape.inv_temp, act_dtype=L.EAT_BF16, expert_dtype=L.EAT_BF16)
              for l in range(n_layers)]
    stack = EatStack(params, B, [to_device(w) for w in w_host],
                     [torch.from_numpy(m).view(torch.bfloat16).cuda() for m in mixes])
    prms = []
    for l in range(n_layers):
        prm = PT.oracle_params(shape, L.MODES[mode], K=caps[l])
        prm.round_h = True
        prms.append(prm)
    return shape, w_host, mixes, stack, prms


def _run(mode, n_layers, d, E, F, B, steps, name, zero_w2=False, caps=None):
    shape, w_host, mixes, stack, prms = _build(mode, n_layers, d, E, F, B, zero_w2=zero_w2, caps=caps)
    accs = [O.zero_accounts(E) for _ in range(n_layers)]
    hs = HiddenStream(shape, B, d=d)
    compared_steps = 0
    ds_h = [0.0] * n_layers           # bound on |S_h(gpu accounts) - S_h(oracle accounts)| per layer
    for step in range(steps):
        x = hs.next()
        masks = torch.empty(n_layers, B, dtype=torch.int64, device="cuda")
        probs = torch.empty(n_layers, B, E, dtype=torch.float32, device="cuda")
        h = stack.forward(torch.from_numpy(x).view(torch.bfloat16).cuda(), masks_out=masks, probs_out=probs)
        torch.cuda.synchronize()
        ref = O.stack_step(x, w_host, mixes, accs, None, prms)
        pg = probs.cpu().numpy()
        taint = np.zeros(B, dtype=bool)
        dps, borders, dp_sum = [], [], []
        for l in range(n_layers):
            r = ref.layers[l].routing
            ok = ~taint
            dp_t = np.abs(pg[l] - r.p).max(axis=1)
            dp = float(dp_t[ok].max()) if ok.any() else 0.0
            assert dp <= DP_CEIL, f"layer {l}: router probabilities differ by {dp:.2e}"
            assert np.median(dp_t) <= DP_MEDIAN, f"layer {l}: median difference {np.median(dp_t):.2e}"
            shift = prms[l].beta * ds_h[l] if mode == "eat" else 0.0
            border = PT.borderline(r, prms[l], eps_b=np.maximum(PT.EPS_B, 4.0 * (dp_t + shift))) & ok
            gm = PT.masks_to_list(masks[l])
            bad = [t for t in range(B) if ok[t] and not border[t] and gm[t] != r.masks[t]]
            assert not bad, f"layer {l}: {len(bad)} mask mismatches outside the per-token band"
            if mode != "topp":
                assert all(bin(int(m)).count("1") <= prms[l].K for m in gm), f"layer {l}: more than K experts"
            taint |= border
            dps.append(dp)
            dp_sum.append(float(dp_t.sum()))
            borders.append(int(border.sum()))
        assert taint.mean() <= MAX_TAINTED[E], f"{taint.sum()} of {B} tokens excluded"
        hg = h.view(torch.int16).cpu().numpy().view(np.uint16)
        err = PT.row_rel_err(O.widen(hg), ref.h)[~taint]
        kmean = [float(np.mean([bin(int(m)).count("1") for m in o.routing.masks])) for o in ref.layers]
        PT.report(f"stack {name} {mode} step {step}", layers=n_layers, T=B, max_dp=f"{max(dps):.1e}",
                  excluded=int(taint.sum()),
                  borderline=borders, max_rel_h=f"{err.max():.2e}" if err.size else "n/a",
                  mean_k=[round(k, 2) for k in kmean])
        assert err.size == 0 or err.max() <= TOL_H
        compared_steps += 1
        if mode == "eat":
            if taint.any():
                break          # a different pick changes that layer's accounts: later steps diverge
            for l, lay in enumerate(stack.layers):
                n, pt, cs = lay.accounts_host()
                rn, rpt, rcs = ref.layers[l].acc
                np.testing.assert_array_equal(n, rn)
                # P_total adds p over the selecting tokens: it can differ by at
                # most the layer's summed |p_gpu - p_oracle| (plus fp32 rounding)
                np.testing.assert_allclose(pt, rpt, rtol=1e-5, atol=dp_sum[l] + 1e-6)
                np.testing.assert_allclose(cs, rcs, rtol=PT.TOL_C_BF16, atol=1e-6)
                nn = np.maximum(n, 1).astype(np.float64)
                ds_h[l] = float(np.max(prms[l].w2 * np.abs(pt.astype(np.float64) - rpt) / nn
                                       + prms[l].w3 * np.abs(cs.astype(np.float64) - rcs)))
        accs = [o.acc for o in ref.layers]
    stack.close()
    assert compared_steps >= 1


@pytest.mark.parametrize("mode", ["eat", "topk", "topp"])
def test_stack_parity_reduced(mode):
    # 4 layers, d=256, 16 experts of width 128, K=8, 32 tokens, 3 steps
    _run(mode, n_layers=4, d=256, E=16, F=128, B=32, steps=3, name="reduced")


@pytest.mark.parametrize("mode", ["eat", "topk"])
def test_stack_parity_zero_expert_output(mode):
    # RMSNorm, routing, residual and mixing through 6 layers, 3 steps
    _run(mode, n_layers=6, d=256, E=16, F=128, B=32, steps=3, name="w2=0", zero_w2=True)


@pytest.mark.parametrize("mode", ["eat", "topk"])
def test_stack_parity_layerwise_caps(mode):
    # layer-wise sparsity: K = 2 in the lower two layers, 8 in the upper two
    from paper_2609_33614_amd.layer import layerwise_caps
    _run(mode, n_layers=4, d=256, E=16, F=128, B=32, steps=2, name="caps 2,2,8,8",
         caps=layerwise_caps(4, 2, 2, 8))


@pytest.mark.parametrize("mode", ["eat", "topk"])
def test_stack_parity_layer_shape(mode):
    # the 16-layer workload's layer shape (d=2048, 64 experts of width 1024,
    # K=8) at its decode batch of 64, two layers, one step
    _run(mode, n_layers=2, d=2048, E=64, F=1024, B=64, steps=1, name="d2048")


@pytest.mark.parametrize("d", [192, 384])
def test_stack_parity_mixing_slices(d):
    # d = 192 leaves the mixing GEMM one reduction slice and d = 384 two (the
    # other cases take four or eight), so every instance of the split-summing
    # RMSNorm pass runs; EAT, 3 layers, 2 steps
    _run("eat", n_layers=3, d=d, E=16, F=128, B=32, steps=2, name=f"d{d}")


def test_stack_reset_clears_every_layer():
    shape, w_host, mixes, stack, prms = _build("eat", 2, 256, 16, 128, 8)
    x = torch.from_numpy(HiddenStream(shape, 8, d=256).next()).view(torch.bfloat16).cuda()
    stack.forward(x)
    torch.cuda.synchronize()
    assert all(lay.accounts_host()[0].sum() > 0 for lay in stack.layers)
    stack.reset_accounts()
    torch.cuda.synchronize()
    assert all(lay.accounts_host()[0].sum() == 0 for lay in stack.layers)
    stack.close()


@pytest.mark.parametrize("mode", ["topk", "eat"])
def test_stack_mixed_expert_counts(mode):
    """Layers with different expert counts (16, 100, 16: one, two and one
    64-bit mask words per token): each layer's masks and probabilities land at
    its own offset of masks_out / probs_out (T * words_l and T * E_l after the
    layers before it), checked layer by layer against the oracle."""
    shape = SHAPES["stack16"]
    Es, d, F, B = [16, 100, 16], 256, 128, 32
    nl = len(Es)
    w_host = [make_layer_weights(shape, layer=l, E=E, d=d, F=F) for l, E in enumerate(Es)]
    mixes = [make_mixing(shape, l, d=d) for l in range(nl)]
    params = [L.eat_params_default(mode=L.MODES[mode], E=E, d_model=d, d_ffn=F, top_k=4, top_p=shape.top_p,
                                   inv_temperature=shape.inv_temp) for E in Es]
    stack = EatStack(params, B, [to_device(w) for w in w_host],
                     [torch.from_numpy(m).view(torch.bfloat16).cuda() for m in mixes])
    prms = []
    for _ in range(nl):
        prm = PT.oracle_params(shape, L.MODES[mode], K=4)
        prm.round_h = True
        prms.append(prm)
    words = [L.mask_words(E) for E in Es]
    x = HiddenStream(shape, B, d=d).next()
    masks = torch.zeros(B * sum(words), dtype=torch.int64, device="cuda")
    probs = torch.zeros(B * sum(Es), dtype=torch.float32, device="cuda")
    h = stack.forward(torch.from_numpy(x).view(torch.bfloat16).cuda(), masks_out=masks, probs_out=probs)
    torch.cuda.synchronize()
    ref = O.stack_step(x, w_host, mixes, [O.zero_accounts(E) for E in Es], None, prms)
    mg, pg = masks.cpu(), probs.cpu().numpy()
    taint = np.zeros(B, dtype=bool)
    moff = poff = 0
    for l, (E, W) in enumerate(zip(Es, words)):
        r = ref.layers[l].routing
        pl = pg[poff:poff + B * E].reshape(B, E)
        ml = mg[moff:moff + B * W].reshape(B, W) if W > 1 else mg[moff:moff + B]
        dp_t = np.abs(pl - r.p).max(axis=1)
        assert float(dp_t[~taint].max()) <= DP_CEIL, f"layer {l}"
        border = PT.borderline(r, prms[l], eps_b=np.maximum(PT.EPS_B, 4.0 * dp_t)) & ~taint
        gm = PT.masks_to_list(ml)
        bad = [t for t in range(B) if not taint[t] and not border[t] and gm[t] != r.masks[t]]
        assert not bad, f"layer {l} (E={E}): {len(bad)} mask mismatches"
        taint |= border
        moff += B * W
        poff += B * E
    assert taint.mean() <= 0.5
    hg = h.view(torch.int16).cpu().numpy().view(np.uint16)
    err = PT.row_rel_err(O.widen(hg), ref.h)[~taint]
    PT.report(f"stack mixed E {mode}", layers=nl, T=B, excluded=int(taint.sum()),
              max_rel_h=f"{err.max():.2e}" if err.size else "n/a")
    assert err.size == 0 or err.max() <= TOL_H
    stack.close()
