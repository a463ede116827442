"""Pin the oracle's routing at more than 64 experts (E = 128, 200, 256).

Masks are Python ints, so experts past bit 63 must land in the right bits;
the selection rules are checked against torch.topk, numpy's quantile and
the characterisations used for small E (a minimal reaching prefix for
Top-P, Top-K on the importance once every expert clears the threshold).
"""
import numpy as np
import pytest
import torch

import oracle as O

WIDE = [128, 200, 256]


def _rows(E, T, seed):
    rng = np.random.default_rng(seed)
    # peaked rows, like a router with a few favoured experts
    return torch.softmax(torch.from_numpy(rng.standard_normal((T, E)) * 2.0), dim=1).numpy()


@pytest.mark.parametrize("E", WIDE)
def test_topk_wide_matches_torch_topk(E):
    p = _rows(E, 40, E)
    r = O.route_probs(p, None, None, O.Params(mode=O.MODE_TOPK, K=8))
    ref = torch.topk(torch.from_numpy(p), 8, dim=1).indices.numpy()
    for t in range(40):
        assert r.masks[t] == sum(1 << int(e) for e in ref[t])
    assert any(m >> 64 for m in r.masks)             # experts past the first word are chosen


@pytest.mark.parametrize("E", WIDE)
@pytest.mark.parametrize("thr", [0.3, 0.6, 0.9])
def test_topp_wide_is_minimal_reaching_prefix(E, thr):
    p = _rows(E, 30, E + 1)
    r = O.route_probs(p, None, None, O.Params(mode=O.MODE_TOPP, top_p=thr))
    for t in range(30):
        sel = r.selected(t)
        k = len(sel)
        # the k largest probabilities (torch.topk), and no shorter set reaches thr
        top = torch.topk(torch.from_numpy(p[t]), k).values.numpy()
        assert sorted(sel) == sorted(torch.topk(torch.from_numpy(p[t]), k).indices.tolist())
        assert p[t][sel].sum() >= thr
        assert k == 1 or top[:k - 1].sum() < thr


@pytest.mark.parametrize("E", WIDE)
def test_quantile_wide_matches_numpy(E):
    rng = np.random.default_rng(E)
    for _ in range(10):
        v = rng.dirichlet(np.ones(E))
        for q in (0.1, 0.9):
            assert O.quantile(v, q) == pytest.approx(np.quantile(v, q, method="linear"), abs=1e-15)


@pytest.mark.parametrize("E", WIDE)
def test_eat_wide_large_history_is_topk_on_importance(E):
    rng = np.random.default_rng(E + 2)
    K = 8
    p = _rows(E, 30, E + 3)
    acc = (np.full(E, 10, np.int64), np.full(E, 5.0, np.float32), (rng.random(E) * 3 + 1).astype(np.float32))
    r = O.route_probs(p, acc, None, O.Params(K=K))
    for t in range(30):
        assert (r.I[t] > r.thr[t]["tau_final"]).all()
        assert r.masks[t] == sum(1 << int(e) for e in torch.topk(torch.from_numpy(r.I[t]), K).indices)


@pytest.mark.parametrize("E", WIDE)
def test_eat_wide_zero_accounts_beta_zero_and_uniform(E):
    rng = np.random.default_rng(E + 4)
    p = _rows(E, 20, E + 5)
    # beta = 0: accounts play no part
    acc = (rng.integers(0, 9, E).astype(np.int64), (rng.random(E) * 4).astype(np.float32),
           (rng.random(E) * 9).astype(np.float32))
    a = O.route_probs(p, acc, None, O.Params(beta=0.0, K=8))
    b = O.route_probs(p, O.zero_accounts(E), None, O.Params(beta=0.0, K=8))
    assert a.masks == b.masks
    # uniform row, empty accounts: no candidate clears tau, argmax takes expert 0
    u = np.full((1, E), 1.0 / E)
    assert O.route_probs(u, O.zero_accounts(E), None, O.Params(K=8)).masks == [1]
    # a favoured expert in the top word is the argmax when nothing clears tau
    acc_top = (np.zeros(E, np.int64), np.zeros(E, np.float32), np.zeros(E, np.float32))
    v = np.full((1, E), 1.0); v[0, E - 1] = 1.5
    v /= v.sum()
    r = O.route_probs(v, acc_top, None, O.Params(K=8))
    assert r.masks[0] >> (E - 1) & 1
