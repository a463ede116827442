"""GPU parity of the stacked-layer step (eat_stack_forward) against the
oracle: per-layer selection masks and router probabilities, the final
hidden rows and every layer's accounts, at every step.

The oracle rounds the experts' hidden activation to bf16 here as the GPU
stores it (reading R27, ``round_h``), and at prefill sizes each expert's
output row too (``round_y``).  What remains is that each side rounds
r, h and u to bf16 from its own value (fp32 on the GPU, fp64 in the
oracle), so an element near a rounding boundary can differ by one bf16 step
and reach the next router.  The borderline band of a token at a layer is
therefore 4x its own largest |p_gpu - p_oracle| there (never below the
single-layer band; that difference itself must stay below the ceiling
below), plus, from the second EAT step on, the bound that the two sides'
slightly different account states put on the history score (Eq. 1-2).
Tokens outside the band must match bit for bit; every token inside it must
carry a valid selection, which the oracle then adopts (``stack_follow``), so
the two sides stay on one path through all layers and steps and every
token's final row and every layer's accounts are compared.

Most tokens never meet a rounding boundary: the median |p_gpu - p_oracle|
over the tokens of every layer must stay at the single-layer level.

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

# |p_gpu - p_oracle| of a token: one bf16 step (2**-8 relative) in an element
# of r or h reaches the next router as ~2.5e-4 relative in u, and such steps
# compound over the layers; a wrong kernel shows up as ~1e-1
DP_CEIL = 2e-3


def dp_median(d: int) -> float:
    """Ceiling of the median of that difference over the tokens of a layer.
    One bf16 step in one element of r moves every element of the next u by
    about 2**-8 / sqrt(d) relative and a router probability by a few 1e-6 at
    d = 2048; a row of d elements meets such a step at one of its three
    rounding points with odds ~ 1e-4 d per layer, so at d = 2048 most tokens
    carry one, while at d <= 512 most carry none."""
    return 1e-6 if d < 1024 else 1e-5
TOL_H = 2e-2          # per-token max|dh| / max|h| after the last layer


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
        prm.round_y = PT.rows_bf16(B, caps[l], E, d, F)
        prms.append(prm)
    return shape, w_host, mixes, stack, prms


def _pick(name, l, r, prm, probs_l, mask_l, shift, stats, d):
    """The routing of layer l as the oracle computes it, checked against the
    GPU's (probabilities, masks outside the band, validity inside it), with
    the GPU's borderline choices adopted."""
    dp_t = np.abs(probs_l - r.p).max(axis=1)
    assert dp_t.max() <= DP_CEIL, f"{name} layer {l}: router probabilities differ by {dp_t.max():.2e}"
    assert np.median(dp_t) <= dp_median(d), f"{name} layer {l}: median difference {np.median(dp_t):.2e}"
    gm = PT.masks_to_list(mask_l)
    border, ra = PT.compare_masks(f"{name} layer {l}", gm, r, prm, np.maximum(PT.EPS_B, 4.0 * dp_t), shift)
    if prm.mode == O.MODE_TOPK:
        assert all(bin(int(m)).count("1") == prm.K for m in gm), f"layer {l}: not K experts"
    stats.setdefault("dp", []).append(float(dp_t.max()))
    stats.setdefault("dp_sum", []).append(float(dp_t.sum()))
    stats.setdefault("borderline", []).append(int(border.sum()))
    return ra


def _run(mode, n_layers, d, E, F, B, steps, name, zero_w2=False, caps=None):
    shape, w_host, mixes, stack, prms = _build(mode, n_layers, d, E, F, B, zero_w2=zero_w2, caps=caps)
    accs = [O.zero_accounts(E) for _ in range(n_layers)]
    hs = HiddenStream(shape, B, d=d)
    total_border = 0
    p_tol = np.zeros(n_layers)         # P_total's difference bound, summed over the steps so far
    for step in range(steps):
        shifts = [PT.history_shift(lay.accounts_host(), a, prm) for lay, a, prm in zip(stack.layers, accs, prms)]
        x = hs.next()
        masks = torch.empty(n_layers, B, dtype=torch.int64, device="cuda")
        probs = torch.empty(n_layers, B, E, dtype=torch.float32, device="cuda")
        h = stack.forward(torch.from_numpy(x).view(torch.bfloat16).cuda(), masks_out=masks, probs_out=probs)
        torch.cuda.synchronize()
        pg, mg = probs.cpu().numpy(), masks.cpu()
        stats = {}
        ref = PT.stack_follow(x, w_host, mixes, accs, prms,
                              lambda l, r: _pick(f"stack {name} {mode} step {step}", l, r, prms[l], pg[l], mg[l],
                                                 shifts[l], stats, d))
        hg = h.view(torch.int16).cpu().numpy().view(np.uint16)
        err = PT.row_rel_err(O.widen(hg), ref.h)
        kmean = [float(np.mean(o.routing.k)) for o in ref.layers]
        total_border += sum(stats["borderline"])
        PT.report(f"stack {name} {mode} step {step}", layers=n_layers, T=B, max_dp=f"{max(stats['dp']):.1e}",
                  borderline_validated=stats["borderline"], max_shift=f"{max(shifts):.1e}",
                  max_rel_h=f"{err.max():.2e}", mean_k=[round(k, 2) for k in kmean])
        assert err.max() <= TOL_H
        if mode == "eat":
            p_tol += np.array(stats["dp_sum"])
            for l, lay in enumerate(stack.layers):
                n, pt, cs = lay.accounts_host()
                rn, rpt, rcs = ref.layers[l].acc
                np.testing.assert_array_equal(n, rn)
                # P_total adds p over the selecting tokens: each step can move
                # it by at most the layer's summed |p_gpu - p_oracle| (plus fp32
                # rounding), and the differences of the steps add up
                np.testing.assert_allclose(pt, rpt, rtol=1e-5, atol=p_tol[l] + 1e-6)
                np.testing.assert_allclose(cs, rcs, rtol=PT.TOL_C_BF16, atol=1e-6)
        accs = [o.acc for o in ref.layers]
    PT.report(f"stack {name} {mode}", steps=steps, borderline_validated_total=total_border)
    stack.close()


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
    # K=8) at its decode batch of 64, two layers, six steps (accounts carried)
    _run(mode, n_layers=2, d=2048, E=64, F=1024, B=64, steps=6, name="d2048")


@pytest.mark.parametrize("mode", ["eat", "topk"])
def test_stack_parity_prefill_sized(mode):
    # 640 tokens: every layer's experts take the wide tiles (T K >= 256 E) and
    # their bf16 rows go through the bf16-row combine with the residual, the
    # mixing GEMM takes the wide tiles too (T >= 384), and the permutation
    # walks several chunks of tokens; two layers, two steps
    _run(mode, n_layers=2, d=256, E=16, F=128, B=640, steps=2, name="prefill-sized")


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
    mg, pg = masks.cpu(), probs.cpu().numpy()
    moff = np.cumsum([0] + [B * W for W in words])
    poff = np.cumsum([0] + [B * E for E in Es])
    stats = {}

    def pick(l, r):
        E, W = Es[l], words[l]
        pl = pg[poff[l]:poff[l] + B * E].reshape(B, E)
        ml = mg[moff[l]:moff[l] + B * W].reshape(B, W) if W > 1 else mg[moff[l]:moff[l] + B]
        return _pick(f"stack mixed E {mode}", l, r, prms[l], pl, ml, 0.0, stats, d)

    ref = PT.stack_follow(x, w_host, mixes, [O.zero_accounts(E) for E in Es], prms, pick)
    hg = h.view(torch.int16).cpu().numpy().view(np.uint16)
    err = PT.row_rel_err(O.widen(hg), ref.h)
    PT.report(f"stack mixed E {mode}", layers=nl, T=B, borderline_validated=stats["borderline"],
              max_rel_h=f"{err.max():.2e}")
    assert err.max() <= TOL_H
    if mode == "eat":
        for l, lay in enumerate(stack.layers):
            n, pt, cs = lay.accounts_host()
            np.testing.assert_array_equal(n, ref.layers[l].acc[0])
            np.testing.assert_allclose(cs, ref.layers[l].acc[2], rtol=PT.TOL_C_BF16, atol=1e-6)
    stack.close()
