"""The library's calls captured in a HIP graph and replayed: every replay
must equal the eager call on the same inputs bit for bit (outputs, masks
and the account state it carries forward).  Replays are interleaved with
eager work and synchronisations, as a serving loop would run them."""
import numpy as np
import pytest
import torch

from paper_2609_33614_amd import _lib as L
from paper_2609_33614_amd.layer import EatLayer, EatStack, capture, to_device
from workload import SHAPES, HiddenStream, make_layer_weights, make_mixing

pytestmark = pytest.mark.gpu


def _same(a: torch.Tensor, b: torch.Tensor) -> bool:
    return torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a,
                       b.view(torch.int16) if b.dtype == torch.bfloat16 else b)


@pytest.mark.parametrize("mode", ["eat", "topk"])
def test_layer_graph_replays_match_eager(mode):
    shape = SHAPES["mixtral"]
    d, F, E, T = 512, 768, 8, 64
    w = to_device(make_layer_weights(shape, E=E, d=d, F=F))
    p = L.eat_params_default(mode=L.MODES[mode], E=E, d_model=d, d_ffn=F, top_k=shape.K,
                             inv_temperature=shape.inv_temp)
    eager, graphed = EatLayer(p, T, w), EatLayer(p, T, w)
    xs = torch.from_numpy(HiddenStream(shape, T, d=d).steps(6)).view(torch.bfloat16).cuda()
    x_in = xs[0].clone()
    y_g = torch.empty(T, d, dtype=torch.bfloat16, device="cuda")
    m_g = torch.empty(T, dtype=torch.int64, device="cuda")
    g = capture(lambda: graphed.forward(x_in, y=y_g, mask_out=m_g))
    eager.reset_accounts()
    graphed.reset_accounts()
    torch.cuda.synchronize()
    for s in range(xs.shape[0]):
        m_e = torch.empty(T, dtype=torch.int64, device="cuda")
        y_e = eager.forward(xs[s], mask_out=m_e)
        torch.cuda.synchronize()
        x_in.copy_(xs[s])
        g.replay()
        torch.cuda.synchronize()
        assert _same(y_g, y_e), f"step {s}: y differs"
        assert torch.equal(m_g, m_e), f"step {s}: masks differ"
        for a, b in zip(graphed.accounts_host(), eager.accounts_host()):
            np.testing.assert_array_equal(a, b)
    eager.close()
    graphed.close()


def test_stack_graph_replays_match_eager():
    shape = SHAPES["stack16"]
    nl, d, E, F, T = 4, 256, 16, 128, 32
    w = [to_device(make_layer_weights(shape, layer=l, E=E, d=d, F=F)) for l in range(nl)]
    mx = [torch.from_numpy(make_mixing(shape, l, d=d)).view(torch.bfloat16).cuda() for l in range(nl)]
    ps = [L.eat_params_default(mode=L.EAT_MODE_EAT, E=E, d_model=d, d_ffn=F, top_k=shape.K) for _ in range(nl)]
    eager, graphed = EatStack(ps, T, w, mx), EatStack(ps, T, w, mx)
    xs = torch.from_numpy(HiddenStream(shape, T, d=d).steps(5)).view(torch.bfloat16).cuda()
    x_in = xs[0].clone()
    h_g = torch.empty(T, d, dtype=torch.bfloat16, device="cuda")
    m_g = torch.empty(nl, T, dtype=torch.int64, device="cuda")
    g = capture(lambda: graphed.forward(x_in, h_out=h_g, masks_out=m_g))
    eager.reset_accounts()
    graphed.reset_accounts()
    torch.cuda.synchronize()
    for s in range(xs.shape[0]):
        m_e = torch.empty(nl, T, dtype=torch.int64, device="cuda")
        h_e = eager.forward(xs[s], masks_out=m_e)
        torch.cuda.synchronize()
        x_in.copy_(xs[s])
        g.replay()
        torch.cuda.synchronize()
        assert _same(h_g, h_e), f"step {s}: h differs"
        assert torch.equal(m_g, m_e), f"step {s}: masks differ"
        for la, lb in zip(graphed.layers, eager.layers):
            for a, b in zip(la.accounts_host(), lb.accounts_host()):
                np.testing.assert_array_equal(a, b)
    eager.close()
    graphed.close()
