"""Packed expert-weight layout (eat_pack_weights, weight_layout = PACKED).

The pack kernel is checked against the layout written out with torch view
and permute operations; a layer on packed weights must then give the same
bits as the same layer on row-major weights (y, masks, accounts), on every
kernel path: decode stream kernels (gated split and unsplit, split-K down),
the always-on expert, the prefill tiles and the stacked layers.  One case is
also checked against the oracle directly.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_33614_amd import _lib as L
from paper_2609_33614_amd.layer import EatLayer, EatStack, pack_weights, to_device
from tests import parity as PT
from workload import SHAPES, HiddenStream, make_accounts, make_layer_weights, make_mixing, make_prefill

pytestmark = pytest.mark.gpu

MODES = {"eat": L.EAT_MODE_EAT, "topk": L.EAT_MODE_TOPK, "topp": L.EAT_MODE_TOPP}


def _reference_pack(w: torch.Tensor) -> torch.Tensor:
    """[g][M][K] -> blocks (g, M/16, K/32), each 64 lanes l = 16 q + i of 8
    elements W[16 rb + i][32 ks + 8 q ..]."""
    g, M, K = w.shape
    v = w.reshape(g, M // 16, 16, K // 32, 4, 8)          # g, rb, i, ks, q, t
    return v.permute(0, 1, 3, 4, 2, 5).contiguous().reshape(g, M, K)


@pytest.mark.parametrize("g,M,K", [(1, 16, 32), (3, 64, 128), (8, 768, 512), (2, 2048, 1024)])
def test_pack_matches_reference_permutation(g, M, K):
    gen = torch.Generator().manual_seed(g * 1000 + M + K)
    w = torch.randn(g, M, K, generator=gen).to(torch.bfloat16).cuda()
    dst = torch.empty_like(w)
    L.eat_pack_weights(w, g, M, K, dst)
    torch.cuda.synchronize()
    assert torch.equal(dst.view(torch.int16), _reference_pack(w).view(torch.int16))


def _pair(shape_name, mode, E, d, F, Fs=0, T=64, K=None):
    shape = SHAPES[shape_name]
    w = make_layer_weights(shape, E=E, d=d, F=F, F_shared=Fs)
    wdev = to_device(w)
    layers = []
    for layout in (L.EAT_LAYOUT_ROWS, L.EAT_LAYOUT_PACKED):
        p = L.eat_params_default(mode=MODES[mode], E=E, d_model=d, d_ffn=F, top_k=shape.K if K is None else K,
                                 top_p=shape.top_p or 0.6, inv_temperature=shape.inv_temp, d_shared=Fs,
                                 weight_layout=layout)
        layers.append(EatLayer(p, T, wdev if layout == L.EAT_LAYOUT_ROWS else pack_weights(wdev)))
    return shape, w, layers


def _same_bits(shape, layers, x_host, acc=None):
    outs = []
    for lay in layers:
        if acc is not None:
            lay.load_accounts(*acc)
        x = torch.from_numpy(np.ascontiguousarray(x_host)).view(torch.bfloat16).cuda()
        mask = lay.mask_tensor(x.shape[0])
        y = lay.forward(x, mask_out=mask)
        torch.cuda.synchronize()
        outs.append((y.view(torch.int16).cpu(), mask.cpu(), lay.accounts_host()))
    (y0, m0, a0), (y1, m1, a1) = outs
    assert torch.equal(m0, m1)
    assert torch.equal(y0, y1)
    for u, v in zip(a0, a1):
        np.testing.assert_array_equal(u, v)


CASES = [
    # decode-sized calls: stream kernels (reduced shapes, several tiles)
    ("mixtral", dict(E=8, d=512, F=768), 64),
    ("finegrained", dict(E=64, d=256, F=256), 200),
    ("qwen3", dict(E=128, d=256, F=256), 33),
    ("shared", dict(E=60, d=256, F=192, Fs=320), 37),
    # prefill-sized calls: wide tiles (routed experts; the always-on expert)
    ("mixtral", dict(E=8, d=512, F=768), 2048),
    ("qwen3", dict(E=128, d=256, F=256), 4096),
    ("shared", dict(E=60, d=256, F=192, Fs=384), 600),
]


@pytest.mark.parametrize("mode", ["eat", "topk", "topp"])
@pytest.mark.parametrize("shape_name,dims,T", CASES)
def test_packed_layer_is_bit_identical(shape_name, dims, T, mode):
    shape, w, layers = _pair(shape_name, mode, T=T, **dims)
    x = make_prefill(shape, tokens=T, seqs=4, d=dims["d"]) if T >= 600 else HiddenStream(shape, T, d=dims["d"]).next()
    acc = make_accounts(dims["E"], seed=T, c_scale=0.05) if mode == "eat" else None
    _same_bits(shape, layers, x, acc)
    for lay in layers:
        lay.close()


@pytest.mark.parametrize("mode", ["eat", "topk"])
def test_packed_stack_is_bit_identical(mode):
    shape = SHAPES["stack16"]
    nl, B, d, E, F = 3, 64, 256, 16, 256
    ws = [to_device(make_layer_weights(shape, layer=l, E=E, d=d, F=F)) for l in range(nl)]
    ms = [torch.from_numpy(make_mixing(shape, l, d=d)).view(torch.bfloat16).cuda() for l in range(nl)]
    outs = []
    for layout in (L.EAT_LAYOUT_ROWS, L.EAT_LAYOUT_PACKED):
        params = [L.eat_params_default(mode=MODES[mode], E=E, d_model=d, d_ffn=F, top_k=4, weight_layout=layout)
                  for _ in range(nl)]
        wl = ws if layout == L.EAT_LAYOUT_ROWS else [pack_weights(w) for w in ws]
        st = EatStack(params, B, wl, ms)
        xs = torch.from_numpy(HiddenStream(shape, B, d=d).steps(3)).view(torch.bfloat16).cuda()
        h = torch.empty(B, d, dtype=torch.bfloat16, device="cuda")
        masks = torch.empty(3, nl, B, dtype=torch.int64, device="cuda")
        for s in range(3):
            st.forward(xs[s], h_out=h, masks_out=masks[s])
        torch.cuda.synchronize()
        outs.append((h.view(torch.int16).cpu(), masks.cpu(), [l.accounts_host() for l in st.layers]))
        st.close()
    assert torch.equal(outs[0][0], outs[1][0])
    assert torch.equal(outs[0][1], outs[1][1])
    for a0, a1 in zip(outs[0][2], outs[1][2]):
        for u, v in zip(a0, a1):
            np.testing.assert_array_equal(u, v)
