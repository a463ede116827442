"""Pins of the oracle's stacked-layer evaluation path (RMSNorm, bf16
rounding, residual + mixing composition) against library routines, closed
forms and invariants; no GPU."""
import numpy as np
import pytest
import torch

import oracle as O
from workload import SHAPES, HiddenStream, make_layer_weights, make_mixing

D, E, F = 64, 8, 32


def test_round_bf16_matches_torch_conversion():
    rng = np.random.default_rng(0)
    v = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-20, 20, 20000),
                        # exact ties between two bf16 neighbours (odd and even mantissas)
                        1.0 + (2 * np.arange(200) + 1) * 2.0 ** -8,
                        -(3.0 + (2 * np.arange(200) + 1) * 2.0 ** -7),
                        [0.0, -0.0, 1e-42, -3e-41, 3.0e38]]).astype(np.float32)
    ref = torch.from_numpy(v).to(torch.bfloat16).to(torch.float64).numpy()
    got = O.round_bf16(v.astype(np.float64))
    np.testing.assert_array_equal(got, ref)


def test_rms_norm_matches_torch():
    rng = np.random.default_rng(1)
    h = rng.standard_normal((16, D))
    h[3] *= 1e-3            # mean square comparable to eps: eps must be in the denominator
    h[5] = 2.5              # constant row -> all ones (up to eps)
    for eps in (1e-6, 1e-2):
        ref = torch.nn.functional.rms_norm(torch.from_numpy(h), (D,), eps=eps).numpy()
        np.testing.assert_allclose(O.rms_norm(h, eps), ref, rtol=1e-12, atol=1e-15)
    assert not np.allclose(O.rms_norm(h, 1e-6)[3], h[3] / np.sqrt(np.mean(h[3] ** 2)), rtol=1e-3)
    # scale invariance
    np.testing.assert_allclose(O.rms_norm(7.0 * h[[0, 1]], 0.0), O.rms_norm(h[[0, 1]], 0.0), rtol=1e-12)


def _stack(L, mode, zero_w2=False, identity_mix=False, seed=0):
    shape = SHAPES["stack16"]
    layers, mixes, prms, accs = [], [], [], []
    for l in range(L):
        w = make_layer_weights(shape, seed=seed, layer=l, E=E, d=D, F=F)
        if zero_w2:
            w["w2"] = np.zeros_like(w["w2"])
        layers.append(w)
        mixes.append(O.round_bf16(np.eye(D)) if identity_mix else make_mixing(shape, l, seed=seed, d=D))
        prms.append(O.Params(mode=mode, K=2, top_p=0.6))
        accs.append(O.zero_accounts(E))
    x = HiddenStream(shape, 12, seed=seed, d=D).next()
    return x, layers, mixes, accs, prms


@pytest.mark.parametrize("mode", [O.MODE_EAT, O.MODE_TOPK])
def test_zero_expert_output_and_identity_mixing_keep_h(mode):
    x, layers, mixes, accs, prms = _stack(3, mode, zero_w2=True, identity_mix=True)
    out = O.stack_step(x, layers, mixes, accs, None, prms)
    np.testing.assert_array_equal(out.h, O.widen(x))


def test_zero_expert_output_applies_the_mixing_chain():
    x, layers, mixes, accs, prms = _stack(3, O.MODE_TOPK, zero_w2=True)
    out = O.stack_step(x, layers, mixes, accs, None, prms)
    chain = O.widen(x)
    for m in mixes:
        chain = chain @ O.widen(m).T
    rel = np.linalg.norm(out.h - chain, axis=1) / np.linalg.norm(chain, axis=1)
    assert rel.max() < 3 * 2.0 ** -8
    # and the product is with M^T: the untransposed chain is far off
    wrong = O.widen(x)
    for m in mixes:
        wrong = wrong @ O.widen(m)
    assert (np.linalg.norm(out.h - wrong, axis=1) / np.linalg.norm(wrong, axis=1)).min() > 0.1


def test_layers_keep_their_own_accounts():
    x, layers, mixes, accs, prms = _stack(3, O.MODE_EAT)
    out = O.stack_step(x, layers, mixes, accs, None, prms)
    h = O.widen(x)
    for l, o in enumerate(out.layers):
        n, pt, cs = o.acc
        assert n.sum() == sum(bin(int(m)).count("1") for m in o.routing.masks)
        # the layer alone, fed the same normalised input, ends in the same state
        u = O.round_bf16(O.rms_norm(h))
        solo = O.moe_step(u, layers[l], O.zero_accounts(E), None, prms[l])
        np.testing.assert_array_equal(solo.acc[0], n)
        np.testing.assert_array_equal(solo.acc[2], cs)
        h = O.round_bf16(O.round_bf16(h + o.y) @ O.widen(mixes[l]).T)
        # layer input RMS is 1 up to bf16 rounding
        assert abs(np.sqrt(np.mean(u * u, axis=1)) - 1).max() < 2 ** -7
    np.testing.assert_array_equal(h, out.h)


def test_topk_layers_select_exactly_k():
    x, layers, mixes, accs, prms = _stack(4, O.MODE_TOPK)
    out = O.stack_step(x, layers, mixes, accs, None, prms)
    for o in out.layers:
        assert all(bin(int(m)).count("1") == 2 for m in o.routing.masks)
