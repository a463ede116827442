"""Closed forms, special cases and invariances of the oracle.

* Eq. 7: the renormalised gates sum to S / (S + eps).
* Eq. 3-5: mu_w = 1/E for a softmax row, so tau <= 1/E; tau_final lies in
  [tau_min, tau_max].
* Sec. 3.2: the EMA after n activations is sum_j alpha (1-alpha)^(n-j) m_j;
  alpha = 1 keeps the last norm, alpha = 0 keeps zero; N is the column sum
  of the masks.
* beta = 0 removes the history; a history that lifts every I above the
  threshold turns EAT into Top-K on I.
* Snapshot semantics: one token per step equals sequential routing;
  permuting tokens inside a step permutes y and leaves the accounts alone.
* Scaling W2 by 2 scales y and C_s by 2 exactly (routing unchanged when
  C_s enters Eq. 1 as a share).
* A one-expert selection gives y = o p / (p + eps); the gather-based layer
  equals a dense sum over all experts weighted by g_norm.
"""
import numpy as np
import pytest

import oracle as O
from workload import SHAPES, HiddenStream, make_layer_weights


def _small_layer(E=8, d=32, F=48, bf16=False, seed=11, shared=0):
    base = SHAPES["tiny"] if not bf16 else SHAPES["finegrained"]
    w = make_layer_weights(base, seed=seed, E=E, d=d, F=F, F_shared=shared)
    return w


def _x(T, d, seed=5, bf16=False):
    shape = SHAPES["finegrained"] if bf16 else SHAPES["tiny"]
    return HiddenStream(shape, T, seed=seed, d=d).next()


def test_gate_sum_closed_form():
    rng = np.random.default_rng(0)
    prm = O.Params(mode=O.MODE_TOPK, K=3)
    p = rng.dirichlet(np.ones(8), size=40)
    r = O.route_probs(p, None, None, prm)
    for t in range(40):
        S = sum(p[t, i] for i in r.selected(t))
        assert r.g_norm[t].sum() == pytest.approx(S / (S + 1e-8), abs=1e-15)
        assert abs(r.g_norm[t].sum() - 1.0) <= 1e-8 / S + 1e-15


def test_threshold_bounds_and_mean():
    rng = np.random.default_rng(1)
    prm = O.Params()
    for E in (4, 8, 64):
        for _ in range(20):
            g = rng.dirichlet(np.ones(E) * 0.3)
            th = O.threshold(g, int(rng.integers(-1, 2)), prm)
            assert th["mu"] == pytest.approx(1.0 / E, abs=1e-15)
            assert th["tau"] <= 1.0 / E + 1e-15
            assert th["tau_min"] <= th["tau_final"] <= th["tau_max"]
            assert th["tau_s"] in (pytest.approx(0.93 * th["tau"]), pytest.approx(1.14 * th["tau"]))


def test_ema_closed_form_and_counts():
    rng = np.random.default_rng(2)
    E, steps = 4, 6
    for alpha in (0.95, 0.5, 1.0, 0.0):
        prm = O.Params(alpha=alpha)
        acc = O.zero_accounts(E)
        masks_hist, norms_hist = [], []
        for s in range(steps):
            T = 3
            masks = [int(m) for m in rng.integers(1, 2 ** E, T)]
            p = rng.dirichlet(np.ones(E), size=T)
            norms = rng.random((T, E)) * 5
            acc = O.account_update(acc, masks, p, norms, prm)
            masks_hist.append(masks); norms_hist.append(norms)
        for i in range(E):
            n = sum(((m >> i) & 1) for ms in masks_hist for m in ms)
            assert acc[0][i] == n
            # per-step mean norms of expert i over the steps it was active
            means = []
            for ms, nr in zip(masks_hist, norms_hist):
                toks = [t for t, m in enumerate(ms) if (m >> i) & 1]
                if toks:
                    means.append(np.mean([nr[t, i] for t in toks]))
            k = len(means)
            closed = sum(alpha * (1 - alpha) ** (k - 1 - j) * means[j] for j in range(k))
            assert float(acc[2][i]) == pytest.approx(closed, rel=2e-6, abs=1e-7)
            if alpha == 1.0 and means:
                assert float(acc[2][i]) == pytest.approx(means[-1], rel=1e-6)
            if alpha == 0.0:
                assert float(acc[2][i]) == 0.0


def test_beta_zero_ignores_history():
    rng = np.random.default_rng(3)
    p = rng.dirichlet(np.ones(8), size=30)
    prm = O.Params(beta=0.0, K=2)
    acc = (np.array([5, 0, 9, 1, 0, 3, 2, 7], np.int64), rng.random(8).astype(np.float32) * 4,
           rng.random(8).astype(np.float32) * 9)
    a = O.route_probs(p, acc, None, prm)
    b = O.route_probs(p, O.zero_accounts(8), None, prm)
    assert a.masks == b.masks


def test_large_history_reduces_to_topk_on_importance():
    rng = np.random.default_rng(4)
    E, K = 8, 3
    p = rng.dirichlet(np.ones(E), size=30)
    prm = O.Params(K=K)
    acc = (np.full(E, 10, np.int64), np.full(E, 5.0, np.float32),
           (rng.random(E) * 3 + 1).astype(np.float32))
    r = O.route_probs(p, acc, None, prm)
    for t in range(30):
        assert (r.I[t] > r.thr[t]["tau_final"]).all()
        assert r.selected(t) == sorted(np.argsort(-r.I[t], kind="stable")[:K].tolist())


@pytest.mark.parametrize("mode", [O.MODE_EAT, O.MODE_TOPK, O.MODE_TOPP])
def test_single_token_snapshot_equals_sequential(mode):
    w = _small_layer()
    x = _x(1, 32)
    prm = O.Params(mode=mode, K=2, top_p=0.5)
    acc = (np.array([3, 1, 0, 0, 2, 0, 1, 0], np.int64), np.full(8, 0.7, np.float32),
           np.linspace(0, 2, 8).astype(np.float32))
    a = O.moe_step(x, w, acc, np.array([1], np.int8), prm)
    b = O.moe_step(x, w, acc, np.array([1], np.int8), prm, sequential=True)
    np.testing.assert_array_equal(a.y, b.y)
    assert a.routing.masks == b.routing.masks
    for u, v in zip(a.acc, b.acc):
        np.testing.assert_array_equal(u, v)


def test_sequential_differs_from_snapshot_only_through_history():
    # With beta = 0 the accounts cannot influence routing, so a multi-token
    # step routes identically either way and ends in the same accounts.
    w = _small_layer()
    x = _x(6, 32)
    prm = O.Params(beta=0.0)
    a = O.moe_step(x, w, O.zero_accounts(8), None, prm)
    b = O.moe_step(x, w, O.zero_accounts(8), None, prm, sequential=True)
    assert a.routing.masks == b.routing.masks
    np.testing.assert_array_equal(a.acc[0], b.acc[0])
    np.testing.assert_allclose(a.acc[1], b.acc[1], rtol=1e-6)


def test_token_permutation_invariance():
    w = _small_layer()
    x = _x(10, 32)
    prm = O.Params()
    acc = (np.array([3, 1, 0, 4, 2, 0, 1, 0], np.int64), np.full(8, 0.7, np.float32),
           np.linspace(0, 2, 8).astype(np.float32))
    perm = np.random.default_rng(0).permutation(10)
    a = O.moe_step(x, w, acc, None, prm)
    b = O.moe_step(x[perm], w, acc, None, prm)
    np.testing.assert_allclose(b.y, a.y[perm], rtol=1e-13, atol=1e-13)
    for u, v in zip(a.acc, b.acc):
        np.testing.assert_array_equal(u, v)


def test_w2_scaling_scales_output_and_contribution():
    w = _small_layer()
    x = _x(8, 32)
    prm = O.Params(cs_mode=1)
    acc = (np.array([3, 1, 0, 4, 2, 0, 1, 0], np.int64), np.full(8, 0.7, np.float32),
           np.linspace(0, 2, 8).astype(np.float32))
    a = O.moe_step(x, w, acc, None, prm)
    w2 = dict(w); w2["w2"] = w["w2"] * np.float32(2.0)
    acc2 = (acc[0], acc[1], acc[2] * np.float32(2.0))
    b = O.moe_step(x, w2, acc2, None, prm)
    assert a.routing.masks == b.routing.masks
    np.testing.assert_array_equal(b.y, 2.0 * a.y)
    np.testing.assert_array_equal(b.acc[2], np.float32(2.0) * a.acc[2])


def test_single_expert_output_and_dense_sum():
    w = _small_layer()
    x = _x(6, 32)
    prm1 = O.Params(mode=O.MODE_TOPK, K=1)
    out = O.moe_step(x, w, None, None, prm1)
    for t in range(6):
        (e,) = out.routing.selected(t)
        o = O.swiglu(x[t:t + 1], w["w1"][e], w["w3"][e], w["w2"][e])[0]
        p = out.routing.p[t, e]
        np.testing.assert_allclose(out.y[t], o * p / (p + 1e-8), rtol=1e-13, atol=1e-13)
    prm = O.Params(mode=O.MODE_TOPP, top_p=0.7)
    out = O.moe_step(x, w, None, None, prm)
    dense = np.zeros_like(out.y)
    for e in range(8):
        dense += out.routing.g_norm[:, e:e + 1] * O.swiglu(x, w["w1"][e], w["w3"][e], w["w2"][e])
    np.testing.assert_allclose(out.y, dense, rtol=1e-12, atol=1e-12)


def test_shared_expert_added_with_unit_weight():
    w = _small_layer(bf16=True, shared=40)
    x = _x(4, 32, bf16=True)
    prm = O.Params(mode=O.MODE_TOPK, K=2, shared=True)
    with_sh = O.moe_step(x, w, None, None, prm).y
    prm.shared = False
    without = O.moe_step(x, w, None, None, prm).y
    np.testing.assert_allclose(with_sh - without, O.swiglu(x, w["ws1"], w["ws3"], w["ws2"]),
                               rtol=1e-10, atol=1e-10)


def test_baseline_modes_leave_accounts_alone():
    w = _small_layer()
    x = _x(5, 32)
    acc = (np.array([3, 1, 0, 4, 2, 0, 1, 0], np.int64), np.full(8, 0.7, np.float32),
           np.linspace(0, 2, 8).astype(np.float32))
    for mode in (O.MODE_TOPK, O.MODE_TOPP):
        out = O.moe_step(x, w, acc, None, O.Params(mode=mode))
        assert out.acc is acc
