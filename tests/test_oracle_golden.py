"""Pin the oracle to a hand-computed worked example (tests/golden/three_step_e4.json).

The fixture's numbers were worked out by hand from Eq. 1-8 and Sec. 3.3 (the
arithmetic is written out in its 'derivation' lines); nothing in it comes
from the oracle.  A dropped term in Eq. 1, a wrong sign in Eq. 5, a swapped
perplexity factor, the wrong quantile position, a non-strict comparison in
Eq. 6 or a mis-ordered EMA each change at least one checked figure.
"""
import json
import os

import numpy as np
import pytest

import oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def fx():
    with open(os.path.join(HERE, "golden", "three_step_e4.json")) as f:
        return json.load(f)


def _prm(fx):
    return O.Params(mode=O.MODE_EAT, K=fx["K"], cs_mode=0)


def test_three_step_sequence(fx):
    prm = _prm(fx)
    tol = fx["tolerance"]
    acc = O.zero_accounts(fx["E"])
    for s in fx["steps"]:
        p = np.array(s["p"])
        th = O.threshold(p, s["trend"], prm)
        for key in ("mu", "sigma", "tau", "tau_ppl", "tau_s", "tau_min", "tau_max", "tau_final"):
            assert th[key] == pytest.approx(s[key], abs=tol), key
        s_h = O.history_score(*acc, prm)
        np.testing.assert_allclose(s_h, s["s_h"], atol=tol)
        I = O.importance(p, s_h, prm.beta)
        np.testing.assert_allclose(I, s["I"], atol=tol)
        cand = [i for i in range(len(p)) if I[i] > th["tau_final"]]
        assert cand == s["candidates"]
        sel = O.select_eat(I, th["tau_final"], prm.K)
        assert sel == s["selected"]
        g = O.renormalise(p, sel, prm.eps)
        np.testing.assert_allclose(g, s["g_norm"], atol=tol)
        # the whole routing entry point agrees with the pieces
        r = O.route_probs(p[None, :], acc, np.array([s["trend"]], np.int8), prm)
        assert r.masks[0] == O.mask_of(s["selected"])
        assert int(r.k[0]) == len(s["selected"])
        norms = np.array(s["norms"])[None, :]
        acc = O.account_update(acc, r.masks, p[None, :], norms, prm)
        np.testing.assert_array_equal(acc[0], s["N"])
        np.testing.assert_allclose(acc[1], s["P"], rtol=1e-6, atol=1e-7)
        np.testing.assert_allclose(acc[2], s["C"], rtol=1e-6, atol=1e-7)


def test_uniform_probabilities_fall_back_to_argmax(fx):
    prm = _prm(fx)
    u = fx["uniform"]
    p = np.array(u["p"])
    th = O.threshold(p, 0, prm)
    assert th["tau_final"] == pytest.approx(u["tau_final"], abs=1e-12)
    r = O.route_probs(p[None, :], O.zero_accounts(4), None, prm)
    assert r.selected(0) == u["selected"]


def test_top_p_examples(fx):
    for case in fx["top_p"]:
        assert O.select_topp(np.array(case["p"]), case["thr"]) == case["selected"]
        prm = O.Params(mode=O.MODE_TOPP, top_p=case["thr"])
        r = O.route_probs(np.array(case["p"])[None, :], None, None, prm)
        assert r.selected(0) == case["selected"]


def test_null_trend_means_otherwise_branch(fx):
    # No perplexity signal takes the "otherwise" (x0.9) branch of Sec. 3.3;
    # a negative trend does the same; only a positive one takes x1.2.
    prm = _prm(fx)
    p = np.array(fx["steps"][1]["p"])
    t_null = O.route_probs(p[None, :], O.zero_accounts(4), None, prm).thr[0]["tau_ppl"]
    t_neg = O.threshold(p, -1, prm)["tau_ppl"]
    t_pos = O.threshold(p, 1, prm)["tau_ppl"]
    tau = O.threshold(p, 0, prm)["tau"]
    assert t_null == pytest.approx(0.9 * tau) and t_neg == pytest.approx(0.9 * tau)
    assert t_pos == pytest.approx(1.2 * tau)


def test_contribution_share_reading(fx):
    c = fx["cs_share"]
    prm = O.Params(cs_mode=1)
    acc = (np.array(c["N"], np.int64), np.array(c["P"], np.float32), np.array(c["C"], np.float32))
    np.testing.assert_allclose(O.history_score(*acc, prm), c["s_h"], atol=1e-6)


def test_ties_go_to_lower_index(fx):
    t = fx["ties"]
    p = np.array(t["p"])
    for K, sel in t["top_k"].items():
        assert O.select_topk(p, int(K)) == sel
    for thr, sel in t["top_p"].items():
        assert O.select_topp(p, float(thr)) == sel
