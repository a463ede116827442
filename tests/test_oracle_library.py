"""Pin the oracle's building blocks to library routines (scipy, numpy, torch).

Softmax, quantile, population std, top-k, SiLU/SwiGLU and the bf16 widening
each reduce to a textbook routine; a transposed operand, a wrong
interpolation position or a biased variance fails here.
"""
import numpy as np
import pytest
import scipy.special
import torch

import oracle as O
from workload import bf16_bits


def test_router_softmax_matches_scipy():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((7, 24)).astype(np.float32)
    w = rng.standard_normal((5, 24)).astype(np.float32)
    for inv_t in (1.0, 2.0):
        ref = scipy.special.softmax((x.astype(np.float64) @ w.astype(np.float64).T) * inv_t, axis=1)
        np.testing.assert_allclose(O.router_probs(x, w, inv_t), ref, rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("E", [4, 8, 60, 64])
def test_quantile_matches_numpy_linear(E):
    rng = np.random.default_rng(E)
    for _ in range(20):
        v = rng.dirichlet(np.ones(E))
        for q in (0.1, 0.9, 0.0, 1.0, 0.5):
            assert O.quantile(v, q) == pytest.approx(np.quantile(v, q, method="linear"), abs=1e-15)


def test_grounding_matches_numpy_population_std():
    rng = np.random.default_rng(1)
    for E in (4, 8, 64):
        g = rng.dirichlet(np.ones(E))
        mu, sigma, tau = O.grounding(g, 0.5, 1.0)
        assert mu == pytest.approx(np.mean(g), abs=1e-15)
        assert sigma == pytest.approx(np.std(g, ddof=0), rel=1e-12)
        assert tau == pytest.approx(max(0.5 * np.mean(g), np.mean(g) - np.std(g)), rel=1e-12)


def test_topk_matches_torch_topk():
    rng = np.random.default_rng(2)
    for E, K in ((8, 2), (64, 8), (60, 4)):
        p = rng.dirichlet(np.ones(E), size=50)
        ref = torch.topk(torch.from_numpy(p), K, dim=1).indices.numpy()
        for t in range(50):
            assert O.select_topk(p[t], K) == sorted(ref[t].tolist())


def test_swiglu_matches_torch_silu_reference():
    # non-square everywhere so that a transposed operand cannot pass
    rng = np.random.default_rng(3)
    n, d, F = 5, 12, 20
    x = rng.standard_normal((n, d))
    w1 = rng.standard_normal((F, d)); w3 = rng.standard_normal((F, d)); w2 = rng.standard_normal((d, F))
    X = torch.from_numpy(x)
    ref = torch.nn.functional.linear(
        torch.nn.functional.silu(torch.nn.functional.linear(X, torch.from_numpy(w1)))
        * torch.nn.functional.linear(X, torch.from_numpy(w3)),
        torch.from_numpy(w2))
    np.testing.assert_allclose(O.swiglu(x, w1, w3, w2), ref.numpy(), rtol=1e-12, atol=1e-12)
    # with the hidden activation rounded to bf16 (torch's conversion goes
    # through fp32; a double-rounding tie is not expected in 100 values)
    hid = (torch.nn.functional.silu(torch.nn.functional.linear(X, torch.from_numpy(w1)))
           * torch.nn.functional.linear(X, torch.from_numpy(w3)))
    ref_r = torch.nn.functional.linear(hid.float().to(torch.bfloat16).double(), torch.from_numpy(w2))
    got_r = O.swiglu(x, w1, w3, w2, round_h=True)
    np.testing.assert_allclose(got_r, ref_r.numpy(), rtol=1e-12, atol=1e-12)
    assert np.abs(got_r - ref.numpy()).max() > 1e-4            # the rounding is really applied


def test_layer_outputs_round_y_rounds_rows_not_norms():
    """R27 at prefill sizes: each expert's output row enters y rounded to
    bf16 (torch's conversion), its norm stays that of the unrounded row."""
    rng = np.random.default_rng(31)
    T, d, F, E = 6, 16, 24, 3
    w = {"w1": rng.standard_normal((E, F, d)), "w3": rng.standard_normal((E, F, d)),
         "w2": rng.standard_normal((E, d, F))}
    x = rng.standard_normal((T, d))
    masks = [0b011, 0b110, 0b101, 0b001, 0b111, 0b010]
    p = rng.random((T, E))
    g = np.zeros((T, E))
    for t, m in enumerate(masks):
        sel = [e for e in range(E) if (m >> e) & 1]
        g[t, sel] = p[t, sel] / p[t, sel].sum()
    r = O.Routing(p=p, masks=masks, k=np.array([bin(m).count("1") for m in masks]), g_norm=g)
    plain = O.layer_outputs(x, w, r, O.Params())
    got = O.layer_outputs(x, w, r, O.Params(round_y=True))
    X = torch.from_numpy(x)
    ref = np.zeros((T, d))
    for e in range(E):
        o = torch.nn.functional.linear(
            torch.nn.functional.silu(torch.nn.functional.linear(X, torch.from_numpy(w["w1"][e])))
            * torch.nn.functional.linear(X, torch.from_numpy(w["w3"][e])), torch.from_numpy(w["w2"][e]))
        ob = o.float().to(torch.bfloat16).double().numpy()
        for t, m in enumerate(masks):
            if (m >> e) & 1:
                ref[t] += g[t, e] * ob[t]
    np.testing.assert_allclose(got.y, ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(got.norms, plain.norms)
    assert np.abs(got.y - plain.y).max() > 1e-4                 # the rounding is really applied


def test_widen_bf16_matches_torch():
    rng = np.random.default_rng(4)
    a = (rng.standard_normal(1000) * 10).astype(np.float32)
    bits = bf16_bits(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(O.widen(bits), ref)


def test_router_softmax_rows_far_apart():
    # each row is shifted by its own maximum: a row whose logits are all far
    # below another row's must still come out as a proper distribution
    x = np.array([[1.0, 0.0], [0.0, 1.0]], np.float32)
    w = np.array([[2000.0, 0.0], [1999.0, 0.0], [0.0, 1.0]], np.float32)
    p = O.router_probs(x, w)
    ref = scipy.special.softmax(x.astype(np.float64) @ w.astype(np.float64).T, axis=1)
    np.testing.assert_allclose(p, ref, rtol=1e-12, atol=1e-300)
    assert np.isfinite(p).all()


def test_opd_reweighting():
    """Sec. 3.5: p' = s p / sum(s p) before selection."""
    rng = np.random.default_rng(11)
    E, T = 8, 200
    p = torch.softmax(torch.from_numpy(rng.standard_normal((T, E))), dim=1).numpy()
    s = rng.uniform(0.25, 4.0, E)
    # unit scales leave every routing decision unchanged
    for mode in (O.MODE_EAT, O.MODE_TOPK, O.MODE_TOPP):
        a = O.route_probs(p, O.zero_accounts(E), None, O.Params(mode=mode, K=2))
        b = O.route_probs(p, O.zero_accounts(E), None, O.Params(mode=mode, K=2, expert_scale=np.ones(E)))
        assert a.masks == b.masks
        np.testing.assert_allclose(a.g_norm, b.g_norm, rtol=1e-15, atol=0)
    # Top-K on the reweighted row is torch.topk of s * p (the renormaliser is a positive factor)
    r = O.route_probs(p, None, None, O.Params(mode=O.MODE_TOPK, K=3, expert_scale=s))
    ref = torch.topk(torch.from_numpy(p * s), 3, dim=1).indices.numpy()
    for t in range(T):
        assert r.masks[t] == sum(1 << int(e) for e in ref[t])
    np.testing.assert_allclose(r.p.sum(axis=1), 1.0, rtol=1e-14)
    np.testing.assert_allclose(r.p, (p * s) / (p * s).sum(axis=1, keepdims=True), rtol=1e-15)
    # a dominant scale forces its expert into every Top-K selection
    big = np.ones(E); big[5] = 1e6
    r2 = O.route_probs(p, None, None, O.Params(mode=O.MODE_TOPK, K=2, expert_scale=big))
    assert all((m >> 5) & 1 for m in r2.masks)
