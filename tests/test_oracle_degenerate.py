"""Oracle pins for the method's degenerate cases (CPU).

One expert (E = 1): the softmax of a single logit is exactly 1, so every
mode selects expert 0 for every token, Eq. 7-8 give g = 1 / (1 + eps), the
layer output is g times that expert's SwiGLU output (checked against torch's
own SiLU and matrix products), and the Sec. 3.2 update has the closed form
N += T, P_total += T, C_s = (1 - alpha) C_s + alpha * mean ||o||.
A cap equal to the expert count (K = E) and Top-P with p = 1 select every
expert in the baselines; EAT's cap then never binds, so its selection is
the candidate set itself (or the argmax when that set is empty).
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
from workload import SHAPES, HiddenStream, make_accounts, make_layer_weights

MODES = [O.MODE_EAT, O.MODE_TOPK, O.MODE_TOPP]


def _torch_swiglu(x, w):
    xt = torch.from_numpy(O.widen(x))
    w1, w3, w2 = (torch.from_numpy(O.widen(w[k][0])) for k in ("w1", "w3", "w2"))
    return (torch.nn.functional.silu(xt @ w1.T) * (xt @ w3.T)) @ w2.T


@pytest.mark.parametrize("shape_name", ["tiny", "mixtral"])
@pytest.mark.parametrize("mode", MODES)
def test_single_expert_closed_form(shape_name, mode):
    shape = SHAPES[shape_name]
    T, d, F = 9, 64, 64
    w = make_layer_weights(shape, E=1, d=d, F=F)
    x = HiddenStream(shape, T, d=d).next()
    prm = O.Params(mode=mode, K=1, top_p=0.6, inv_temp=shape.inv_temp)
    acc = make_accounts(1, seed=5, c_scale=0.05) if mode == O.MODE_EAT else None
    out = O.moe_step(x, w, acc, None, prm)
    r = out.routing
    assert r.masks == [1] * T and (r.k == 1).all()
    assert (r.p == 1.0).all()
    g = 1.0 / (1.0 + prm.eps)
    np.testing.assert_allclose(r.g_norm[:, 0], g, rtol=0, atol=1e-15)
    o = _torch_swiglu(x, w).numpy()
    np.testing.assert_allclose(out.y, g * o, rtol=1e-12, atol=1e-12)
    if mode == O.MODE_EAT:
        n0, p0, c0 = acc
        n1, p1, c1 = out.acc
        assert int(n1[0]) == int(n0[0]) + T
        assert float(p1[0]) == np.float32(float(p0[0]) + T)
        mean_norm = math.fsum(np.linalg.norm(o, axis=1)) / T
        exp_c = np.float32((1 - prm.alpha) * float(c0[0]) + prm.alpha * mean_norm)
        assert abs(float(c1[0]) - float(exp_c)) <= 2 * np.spacing(np.float32(exp_c))


@pytest.mark.parametrize("E", [4, 8])
def test_cap_equal_to_expert_count(E):
    shape = SHAPES["tiny"]
    T = 16
    w = make_layer_weights(shape, E=E)
    x = HiddenStream(shape, T).next()
    full = (1 << E) - 1
    # baselines: K = E and p = 1 keep every expert
    for prm in (O.Params(mode=O.MODE_TOPK, K=E, inv_temp=shape.inv_temp),
                O.Params(mode=O.MODE_TOPP, K=E, top_p=1.0, inv_temp=shape.inv_temp)):
        r = O.route(x, w["w_router"], None, None, prm)
        assert r.masks == [full] * T and (r.k == E).all()
        np.testing.assert_allclose(r.g_norm.sum(axis=1), 1.0, atol=1e-7)
    # EAT with the cap at E: the candidate set {I > tau_final}, or the argmax
    prm = O.Params(mode=O.MODE_EAT, K=E, inv_temp=shape.inv_temp)
    acc = make_accounts(E, seed=11, c_scale=0.05)
    r = O.route(x, w["w_router"], acc, None, prm)
    for t in range(T):
        tau = r.thr[t]["tau_final"]
        cand = [i for i in range(E) if r.I[t, i] > tau]
        exp = cand if cand else [int(np.argmax(r.I[t]))]
        assert r.selected(t) == exp, t
