"""GPU parity of the perplexity signal (eat_ppl_trend) against the oracle's
ppl_update over several tokens per sequence: NLL, running state and trend.

The GPU's logits are fp32 sums of bf16 products, the oracle's fp64, so the
NLL differs by ~1e-5; a trend is compared wherever the oracle's perplexity
moved by more than TREND_BAND (relative) since the previous token, which
that difference cannot flip.  The LM-head output also feeds one EAT layer's
next step as its ppl_trend, checked against the oracle fed the oracle's
own trend."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_33614_amd import _lib as L
from paper_2609_33614_amd.layer import EatLayer, PplSignal, to_device
from tests import parity as PT
from workload import SHAPES, HiddenStream, make_layer_weights, make_targets, make_vocab_head

pytestmark = pytest.mark.gpu

TOL_NLL = 2e-4
TREND_BAND = 1e-4


@pytest.mark.parametrize("S,d,V,steps", [(64, 512, 32000, 6), (37, 256, 1024, 5), (512, 256, 4096, 3)])
def test_ppl_signal_parity(S, d, V, steps):
    shape = SHAPES["mixtral"]
    w = make_vocab_head(d, V, seed=V)
    sig = PplSignal(S, torch.from_numpy(w).view(torch.bfloat16).cuda())
    sig.reset()
    st = O.ppl_zero_state(S)
    hs = HiddenStream(shape, S, d=d)
    compared = 0
    for step in range(steps):
        h = hs.next()
        y = make_targets(S, V, seed=1000 * step + S)
        tr = sig.step(torch.from_numpy(h).view(torch.bfloat16).cuda(), torch.from_numpy(y).cuda())
        torch.cuda.synchronize()
        prev = st.ppl_prev.copy()
        nll, ppl, trend, st = O.ppl_update(h, w, y, st)
        np.testing.assert_allclose(sig.nll.cpu().numpy(), nll, rtol=0, atol=TOL_NLL)
        np.testing.assert_array_equal(sig.count.cpu().numpy(), st.count)
        np.testing.assert_allclose(sig.nll_sum.cpu().numpy(), st.nll_sum, rtol=0, atol=TOL_NLL * (step + 1))
        clear = (st.count == 1) | (np.abs(ppl - prev) > TREND_BAND * ppl)
        g = tr.cpu().numpy()
        assert (g[clear] == trend[clear]).all(), f"step {step}: trend differs"
        compared += int(clear.sum())
        PT.report(f"ppl S={S} V={V} step {step}", max_dnll=f"{np.abs(sig.nll.cpu().numpy() - nll).max():.1e}",
                  trends_compared=int(clear.sum()), rising=int((trend > 0).sum()))
    assert compared >= S * steps * 0.9


def test_ppl_out_of_range_target_is_nan():
    S, d, V = 8, 128, 256
    w = make_vocab_head(d, V, seed=1)
    sig = PplSignal(S, torch.from_numpy(w).view(torch.bfloat16).cuda())
    sig.reset()
    h = torch.from_numpy(HiddenStream(SHAPES["mixtral"], S, d=d).next()).view(torch.bfloat16).cuda()
    y = torch.tensor([0, 1, -1, V, 5, 6, 7, V + 100], dtype=torch.int32, device="cuda")
    sig.step(h, y)
    torch.cuda.synchronize()
    nll = sig.nll.cpu().numpy()
    assert np.isnan(nll[[2, 3, 7]]).all() and np.isfinite(nll[[0, 1, 4, 5, 6]]).all()


def test_ppl_trend_drives_the_next_step():
    """One EAT layer's second decode step takes the trend the LM head
    produced from its first step's output.  The oracle stores H as bf16
    like the GPU (round_h) and feeds its own signal from its own output;
    tokens whose perplexity change is within TREND_BAND may get either
    trend and are left out of the second step's comparison."""
    shape = SHAPES["mixtral"]
    d, F, E, S, V = 512, 768, 8, 64, 4096
    wl = make_layer_weights(shape, E=E, d=d, F=F)
    p = L.eat_params_default(mode=L.EAT_MODE_EAT, E=E, d_model=d, d_ffn=F, top_k=shape.K,
                             inv_temperature=shape.inv_temp)
    lay = EatLayer(p, S, to_device(wl))
    wv = make_vocab_head(d, V, seed=3)
    sig = PplSignal(S, torch.from_numpy(wv).view(torch.bfloat16).cuda())
    sig.reset()
    prm = PT.oracle_params(shape, L.EAT_MODE_EAT)
    prm.round_h = True
    st = O.ppl_zero_state(S)
    hs = HiddenStream(shape, S, d=d)
    # two tokens per sequence before the routed step, so the trend is defined
    x0, x1, x2 = hs.next(), hs.next(), hs.next()
    acc = O.zero_accounts(E)
    keep = np.ones(S, dtype=bool)
    trend_o = None
    for step, x in enumerate((x0, x1)):
        mask = torch.empty(S, dtype=torch.int64, device="cuda")
        y_dev = lay.forward(torch.from_numpy(x).view(torch.bfloat16).cuda(), mask_out=mask)
        ref = O.moe_step(x, wl, acc, None, prm)
        border = PT.borderline(ref.routing, prm)
        assert not border.any(), "choose inputs without borderline tokens"
        gm = PT.masks_to_list(mask)
        assert gm == list(ref.routing.masks), f"step {step}"
        acc = ref.acc
        tgt = make_targets(S, V, seed=step)
        sig.step(y_dev, torch.from_numpy(tgt).cuda())
        torch.cuda.synchronize()
        prev = st.ppl_prev.copy()
        _, ppl, trend_o, st = O.ppl_update(O.round_bf16(ref.y), wv, tgt, st)
        keep &= (st.count == 1) | (np.abs(ppl - prev) > TREND_BAND * ppl)
    g = sig.trend.cpu().numpy()
    assert (g[keep] == trend_o[keep]).all()
    assert (trend_o[keep] > 0).any() and (trend_o[keep] < 0).any()
    # the routed step: the trend of a sequence whose perplexity change lies
    # within the band may legitimately differ; there the oracle takes the
    # GPU's (either value is a correct trend), everywhere else its own
    trend_g = sig.trend.clone()
    mask = torch.empty(S, dtype=torch.int64, device="cuda")
    lay.forward(torch.from_numpy(x2).view(torch.bfloat16).cuda(), trend=trend_g, mask_out=mask)
    torch.cuda.synchronize()
    trend_use = np.where(keep, trend_o, trend_g.cpu().numpy()).astype(np.int8)
    ref = O.moe_step(x2, wl, acc, trend_use, prm)
    border, _ = PT.compare_masks("ppl -> routing", PT.masks_to_list(mask), ref.routing, prm, PT.EPS_B)
    cmp = keep & ~border
    assert cmp.mean() > 0.8
    PT.report("ppl -> routing", compared=int(cmp.sum()), rising=int((trend_o > 0).sum()))
    lay.close()
