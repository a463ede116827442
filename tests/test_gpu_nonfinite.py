"""Non-finite hidden states (reading R25): a token whose row holds NaN or Inf
gets NaN router scores; its selection follows the documented rule of each
mode and never exceeds what the workspace holds, and every other token of the
call is unaffected -- its mask is identical to a call without the bad
tokens and its output row finite and equal to that call's: bit for bit in
EAT mode, where the bad tokens select nothing and the experts in use are the
same, to the bf16 tolerance in the baselines, where the bad tokens' experts
join the call's and so may change the number of reduction slices the
expert kernels take (an order of additions); and the EAT accounts equal
those of a call with the bad tokens removed (snapshot semantics: tokens are
independent)."""
import numpy as np
import pytest
import torch

from paper_2609_33614_amd import _lib as L
from paper_2609_33614_amd.layer import EatLayer, to_device
from tests import parity as PT
from workload import SHAPES, HiddenStream, bf16_bits, make_accounts, make_layer_weights

pytestmark = pytest.mark.gpu

MODES = {"eat": L.EAT_MODE_EAT, "topk": L.EAT_MODE_TOPK, "topp": L.EAT_MODE_TOPP}
BAD = {3: np.nan, 10: np.inf, 11: -np.inf}


def _bf16_rows(x_bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x_bits)).view(torch.bfloat16).cuda()


def _layer(shape_name, E, d, F, mode, T):
    shape = SHAPES[shape_name]
    w = make_layer_weights(shape, E=E, d=d, F=F)
    p = L.eat_params_default(mode=MODES[mode], E=E, d_model=d, d_ffn=F, top_k=shape.K,
                             top_p=shape.top_p or 0.6, inv_temperature=shape.inv_temp)
    return shape, EatLayer(p, T, to_device(w))


def _run(lay, x, acc):
    if acc is not None:
        lay.load_accounts(*acc)
    mask = lay.mask_tensor(x.shape[0])
    y = lay.forward(x, mask_out=mask)
    torch.cuda.synchronize()
    return y.view(torch.int16).cpu(), PT.masks_to_list(mask), lay.accounts_host()


@pytest.mark.parametrize("mode", ["eat", "topk", "topp"])
@pytest.mark.parametrize("shape_name,E,d,F", [("finegrained", 64, 256, 256), ("qwen3", 128, 256, 256)])
def test_nonfinite_tokens_are_contained(shape_name, E, d, F, mode):
    T = 37
    shape, lay = _layer(shape_name, E, d, F, mode, T)
    good = HiddenStream(shape, T, d=d, seed=5).next()                       # bf16 bits
    bad = good.copy()
    for t, v in BAD.items():
        bad[t] = bf16_bits(np.full(d, v, dtype=np.float32))
    acc = make_accounts(E, seed=9, c_scale=0.05) if mode == "eat" else None

    yb, mb, ab = _run(lay, _bf16_rows(bad), acc)
    yg, mg, ag = _run(lay, _bf16_rows(good), acc)
    keep = [t for t in range(T) if t not in BAD]
    for t in keep:
        assert mb[t] == mg[t], t
        if mode == "eat":
            assert torch.equal(yb[t], yg[t]), t
        else:
            fb = yb[t].view(torch.bfloat16).float()
            fg = yg[t].view(torch.bfloat16).float()
            assert torch.isfinite(fb).all(), t
            assert (fb - fg).abs().max() <= PT.TOL_Y_BF16 * fg.abs().max(), t
    K = shape.K
    for t in BAD:
        k = bin(mb[t]).count("1")
        if mode == "eat":
            assert k == 0                       # no importance beats a NaN threshold, no maximiser
            assert not yb[t].any()              # no expert: y = 0
        elif mode == "topk":
            assert mb[t] == (1 << K) - 1        # ranks collapse to 0: the K lowest indices are kept
        else:
            assert k == E                       # the running sum never reaches p: every expert
    if mode == "eat":
        # the bad tokens select nothing: the accounts equal a call without them
        _, _, a_removed = _run(lay, _bf16_rows(good[keep]), acc)
        for u, v in zip(ab, a_removed):
            np.testing.assert_array_equal(u, v)
    lay.close()
