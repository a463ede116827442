"""CPU checks of the parity rules that judge the GPU's selections.

A borderline token has several correct selections, so the GPU tests accept
any mask that ``parity.valid_choice`` accepts.  These tests pin that rule on
the oracle's own routing (E = 8 and 64, three modes, with and without
history): the oracle's mask is always valid, and for tokens the band does
not reach, every mask one plausible mistake away (an expert dropped, one
added, one swapped for another) is rejected -- so a selector bug shows even
where a test falls back to the validity rule.  ``adopt`` keeps the oracle's
gates for the masks it keeps and renormalises the adopted ones (Eq. 7-8).
"""
import numpy as np
import pytest

import oracle as O
from tests import parity as PT
from workload import make_accounts


def _routing(mode, E, K, T, seed, hist):
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((T, E)) * 1.5
    p = np.exp(z - z.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    prm = O.Params(mode=mode, K=K, top_p=0.6)
    acc = make_accounts(E, seed=seed, c_scale=0.05) if hist else O.zero_accounts(E)
    return O.route_probs(p, acc, None, prm), prm


def _neighbours(m, E):
    on = [e for e in range(E) if (m >> e) & 1]
    off = [e for e in range(E) if not (m >> e) & 1]
    out = [m & ~(1 << e) for e in on if len(on) > 1]
    out += [m | (1 << e) for e in off]
    out += [(m & ~(1 << a)) | (1 << b) for a in on for b in off]
    return out


CASES = [(O.MODE_EAT, 8, 2, False), (O.MODE_EAT, 8, 2, True), (O.MODE_EAT, 64, 8, True),
         (O.MODE_TOPK, 8, 2, False), (O.MODE_TOPK, 64, 8, False), (O.MODE_TOPP, 8, 2, False),
         (O.MODE_TOPP, 64, 8, False)]


@pytest.mark.parametrize("mode,E,K,hist", CASES)
def test_oracle_masks_valid_and_mistakes_rejected(mode, E, K, hist):
    r, prm = _routing(mode, E, K, 60, seed=E + 10 * K + mode, hist=hist)
    border = PT.borderline(r, prm, eps_b=PT.EPS_B)
    checked = 0
    for t in range(len(r.masks)):
        assert PT.valid_choice(r.masks[t], r, t, prm, PT.EPS_B) == "", t
        if border[t]:
            continue
        for m in _neighbours(r.masks[t], E)[:40]:
            assert PT.valid_choice(m, r, t, prm, PT.EPS_B) != "", (t, hex(m))
            checked += 1
    assert checked > 100


def test_eat_near_tie_accepts_both_answers():
    # K = 1: two candidates whose importance differs by less than the band
    E, K = 4, 1
    p = np.array([[0.40, 0.40 + 2e-7, 0.15, 0.05 - 2e-7]])
    prm = O.Params(mode=O.MODE_EAT, K=K)
    r = O.route_probs(p, O.zero_accounts(E), None, prm)
    assert PT.borderline(r, prm, eps_b=PT.EPS_B)[0]
    for m in (0b01, 0b10):
        assert PT.valid_choice(m, r, 0, prm, PT.EPS_B) == ""
    # an exact tie at the K-th value keeps both (the literal rank rule), so
    # within the band that answer is correct too
    assert PT.valid_choice(0b11, r, 0, prm, PT.EPS_B) == ""
    assert PT.valid_choice(0b100, r, 0, prm, PT.EPS_B) != ""
    assert PT.valid_choice(0b101, r, 0, prm, PT.EPS_B) != ""


def test_eat_threshold_straddle_accepts_with_and_without():
    # an importance within the band of tau_final: the candidate may or may
    # not be in the set (|set| <= K), nothing else may change
    E, K = 8, 3
    p = np.array([[0.30, 0.25, 0.12, 0.11, 0.08, 0.07, 0.04, 0.03]])
    prm = O.Params(mode=O.MODE_EAT, K=K)
    r = O.route_probs(p, O.zero_accounts(E), None, prm)
    tf = r.thr[0]["tau_final"]
    # move expert 2's probability onto the threshold (I = (1 - beta) p)
    p2 = p.copy()
    p2[0, 2] = tf / (1 - prm.beta) + 1e-8
    p2[0, 7] -= p2[0, 2] - p[0, 2]
    r2 = O.route_probs(p2, O.zero_accounts(E), None, prm)
    assert PT.borderline(r2, prm, eps_b=PT.EPS_B)[0]
    base = r2.masks[0]
    other = base ^ (1 << 2)
    assert PT.valid_choice(base, r2, 0, prm, PT.EPS_B) == ""
    assert PT.valid_choice(other, r2, 0, prm, PT.EPS_B) == ""
    assert PT.valid_choice(other ^ (1 << 0), r2, 0, prm, PT.EPS_B) != ""


def test_topp_rules():
    prm = O.Params(mode=O.MODE_TOPP, top_p=0.6)
    p = np.array([[0.5, 0.3, 0.15, 0.05]])
    r = O.route_probs(p, None, None, prm)
    assert r.masks[0] == 0b11
    assert PT.valid_choice(0b11, r, 0, prm, PT.EPS_B) == ""
    assert "reach" in PT.valid_choice(0b01, r, 0, prm, PT.EPS_B)
    assert "earlier" in PT.valid_choice(0b111, r, 0, prm, PT.EPS_B)
    assert "outweighs" in PT.valid_choice(0b101, r, 0, prm, PT.EPS_B)
    capped = O.Params(mode=O.MODE_TOPP, top_p=0.95, top_p_cap=2)
    rc = O.route_probs(p, None, None, capped)
    assert rc.masks[0] == 0b11 and PT.valid_choice(0b11, rc, 0, capped, PT.EPS_B) == ""
    assert PT.valid_choice(0b111, rc, 0, capped, PT.EPS_B) != ""


def test_adopt_keeps_oracle_gates_and_renormalises_adopted():
    r, prm = _routing(O.MODE_EAT, 8, 2, 10, seed=3, hist=True)
    border = np.zeros(10, dtype=bool)
    border[4] = True
    gm = list(r.masks)
    gm[4] = 1 << int(np.argmax(r.p[4]))
    a = PT.adopt(r, gm, border, prm)
    assert a.masks[4] == gm[4] and a.k[4] == 1
    np.testing.assert_allclose(a.g_norm[4].sum(), 1.0, rtol=1e-7)
    keep = ~border
    np.testing.assert_array_equal(a.g_norm[keep], r.g_norm[keep])
    assert [a.masks[t] for t in np.flatnonzero(keep)] == [r.masks[t] for t in np.flatnonzero(keep)]


def test_band_for():
    assert PT.band_for(0.0) == PT.EPS_B
    assert PT.band_for(1e-6) == pytest.approx(4e-6)


def test_stack_follow_without_hook_is_the_oracle_stack_step():
    from workload import SHAPES, HiddenStream, make_layer_weights, make_mixing
    shape = SHAPES["stack16"]
    d, E, F, B, nl = 128, 16, 64, 8, 3
    ws = [make_layer_weights(shape, layer=l, E=E, d=d, F=F) for l in range(nl)]
    ms = [make_mixing(shape, l, d=d) for l in range(nl)]
    for mode in (O.MODE_EAT, O.MODE_TOPK):
        prms = [O.Params(mode=mode, K=4, round_h=True) for _ in range(nl)]
        accs = [make_accounts(E, seed=l, c_scale=0.05) for l in range(nl)]
        x = HiddenStream(shape, B, d=d).next()
        a = O.stack_step(x, ws, ms, accs, None, prms)
        b = PT.stack_follow(x, ws, ms, accs, prms, lambda l, r: r)
        np.testing.assert_array_equal(a.h, b.h)
        for la, lb in zip(a.layers, b.layers):
            assert la.routing.masks == lb.routing.masks
            np.testing.assert_array_equal(la.y, lb.y)
            for u, v in zip(la.acc, lb.acc):
                np.testing.assert_array_equal(u, v)
