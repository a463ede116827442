"""Pins of the oracle's perplexity signal: library cross-entropy, closed
forms and a hand-made sequence; no GPU."""
import numpy as np
import torch

import oracle as O


def test_nll_is_torch_cross_entropy():
    rng = np.random.default_rng(5)
    S, d, V = 6, 24, 50
    h = rng.standard_normal((S, d)); w = rng.standard_normal((V, d)) / np.sqrt(d)
    y = rng.integers(0, V, S)
    nll, ppl, trend, st = O.ppl_update(h, w, y, O.ppl_zero_state(S))
    ref = torch.nn.functional.cross_entropy(torch.from_numpy(h @ w.T), torch.from_numpy(y), reduction="none")
    np.testing.assert_allclose(nll, ref.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(ppl, np.exp(nll), rtol=1e-12)
    assert (trend == 0).all() and (st.count == 1).all()


def test_uniform_logits_give_perplexity_v():
    S, d, V = 3, 8, 40
    h = np.zeros((S, d)); w = np.ones((V, d))
    _, ppl, _, _ = O.ppl_update(h, w, [0, 7, 39], O.ppl_zero_state(S))
    np.testing.assert_allclose(ppl, V, rtol=1e-12)


def test_trend_follows_the_running_perplexity():
    # one sequence, logits built so that the NLLs are 1, 2, 0.5, 0.5:
    # running ppl e^1, e^1.5, e^(3.5/3), e^1  -> trend 0, +1, -1, -1
    V = 2
    def step(target_nll, st):
        # two logits a, 0 with target 0: nll = log(1 + e^-a)... solve a for the wanted nll
        a = -np.log(np.exp(target_nll) - 1.0)
        h = np.array([[a]]); w = np.array([[1.0], [0.0]])
        return O.ppl_update(h, w, [0], st)
    st = O.ppl_zero_state(1)
    trends, ppls = [], []
    for want in (1.0, 2.0, 0.5, 0.5):
        nll, ppl, tr, st = step(want, st)
        np.testing.assert_allclose(nll, [want], rtol=1e-12)
        trends.append(int(tr[0])); ppls.append(float(ppl[0]))
    assert trends == [0, 1, -1, -1]
    np.testing.assert_allclose(ppls, np.exp([1.0, 1.5, 3.5 / 3, 1.0]), rtol=1e-12)
    assert st.count[0] == 4
