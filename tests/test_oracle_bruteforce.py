"""Pin the oracle's selection rules by exhaustive enumeration on E <= 8.

Each rule is re-derived here from a different characterisation than the one
the oracle uses (subset enumeration instead of counting / sorting), so an
off-by-one, a flipped inequality or a wrong tie rule fails.
"""
import itertools

import numpy as np
import pytest

import oracle as O


def _vectors(E, rng):
    out = [rng.dirichlet(np.ones(E)) for _ in range(30)]
    out.append(np.full(E, 1.0 / E))                       # uniform
    oh = np.full(E, 1e-3); oh[rng.integers(E)] = 1.0      # near one-hot
    out.append(oh / oh.sum())
    t = rng.dirichlet(np.ones(E)); t[1] = t[0]             # a tie
    out.append(t / t.sum())
    return out


def _brute_eq6(I, tau, K):
    """Eq. 6 by enumeration: among candidates (I > tau), look at every
    K-subset and take the largest achievable sum of I; the K-th value v is
    the smallest member of such a best subset; the final set is every
    candidate with I >= v.  With no candidate: the lowest-index maximiser."""
    E = len(I)
    cand = [i for i in range(E) if I[i] > tau]
    if not cand:
        m = max(I)
        return [min(i for i in range(E) if I[i] == m)]
    if len(cand) <= K:
        return cand
    best, v = -np.inf, None
    for sub in itertools.combinations(cand, K):
        s = sum(I[i] for i in sub)
        if s > best:
            best, v = s, min(I[i] for i in sub)
        elif s == best:
            v = max(v, min(I[i] for i in sub))
    return [i for i in cand if I[i] >= v]


@pytest.mark.parametrize("E", [2, 3, 4, 6, 8])
@pytest.mark.parametrize("K", [1, 2, 3])
def test_eq6_matches_enumeration(E, K):
    if K > E:
        pytest.skip("K > E")
    rng = np.random.default_rng(100 * E + K)
    for p in _vectors(E, rng):
        I = np.round(p * 7, 6)               # rounded so exact ties do occur
        # thresholds equal to some I_i check that the comparison is strict
        for tau in (0.0, 0.5 / E, 1.0 / E, 2.0 / E, 2.0, *sorted(set(I.tolist()))):
            assert O.select_eat(I, tau, K) == _brute_eq6(I, tau, K)


def test_eq6_keeps_all_ties_at_kth_value():
    I = np.array([0.9, 0.5, 0.5, 0.5, 0.1])
    assert O.select_eat(I, 0.2, 2) == [0, 1, 2, 3]


@pytest.mark.parametrize("E", [2, 4, 5, 8])
@pytest.mark.parametrize("K", [1, 2, 4])
def test_topk_is_best_k_subset(E, K):
    if K > E:
        pytest.skip("K > E")
    rng = np.random.default_rng(7 * E + K)
    for p in _vectors(E, rng):
        best, best_sub = -np.inf, None
        for sub in itertools.combinations(range(E), K):   # lexicographic order
            s = sum(p[i] for i in sub)
            if s > best + 1e-15:
                best, best_sub = s, list(sub)
        got = O.select_topk(p, K)
        assert len(got) == K
        assert sum(p[i] for i in got) == pytest.approx(best, abs=1e-15)
        if len(set(np.round(p, 15))) == E:
            assert got == best_sub


@pytest.mark.parametrize("E", [2, 4, 6, 8])
@pytest.mark.parametrize("thr", [0.2, 0.5, 0.6, 0.9, 1.0])
def test_topp_is_smallest_reaching_subset(E, thr):
    rng = np.random.default_rng(E + int(100 * thr))
    for p in _vectors(E, rng)[:30]:                # distinct values only
        got = O.select_topp(p, thr)
        reaching = [s for r in range(1, E + 1) for s in itertools.combinations(range(E), r)
                    if sum(p[i] for i in s) >= thr]
        if not reaching:
            # rounding left the total below thr: every expert is taken
            assert got == list(range(E))
            continue
        size = min(len(s) for s in reaching)
        best = max(sum(p[i] for i in s) for s in reaching if len(s) == size)
        assert len(got) == size
        assert sum(p[i] for i in got) == pytest.approx(best, abs=1e-15)


def test_topp_cap_limits_prefix():
    p = np.array([0.3, 0.25, 0.2, 0.15, 0.1])
    assert O.select_topp(p, 0.9) == [0, 1, 2, 3]
    assert O.select_topp(p, 0.9, cap=2) == [0, 1]


@pytest.mark.parametrize("E", [3, 5, 8])
@pytest.mark.parametrize("thr", [0.5, 0.9])
def test_topp_cap_is_the_heaviest_subset_of_the_capped_size(E, thr):
    # with a cap c the nucleus is the heaviest subset of size min(k*, c),
    # k* the size of the smallest subset reaching thr (by enumeration)
    rng = np.random.default_rng(10 * E + int(10 * thr))
    for p in _vectors(E, rng)[:20]:
        reaching = [s for r in range(1, E + 1) for s in itertools.combinations(range(E), r)
                    if sum(p[i] for i in s) >= thr]
        k_star = min(len(s) for s in reaching) if reaching else E
        for cap in range(1, E + 1):
            size = min(k_star, cap)
            heaviest = max(itertools.combinations(range(E), size), key=lambda s: sum(p[i] for i in s))
            assert O.select_topp(p, thr, cap) == sorted(heaviest), (cap, p)


@pytest.mark.parametrize("E", [4, 8])
def test_eat_route_against_enumeration_with_history(E):
    """Whole per-token EAT path with random non-zero accounts: the oracle's
    selection equals the enumerated Eq. 6 on its own I and tau_final."""
    rng = np.random.default_rng(E)
    prm = O.Params(K=2)
    acc = (rng.integers(0, 50, E).astype(np.int64),
           rng.random(E).astype(np.float32) * 10, rng.random(E).astype(np.float32))
    p = np.stack(_vectors(E, rng))
    r = O.route_probs(p, acc, None, prm)
    for t in range(p.shape[0]):
        assert r.selected(t) == _brute_eq6(r.I[t], r.thr[t]["tau_final"], prm.K)
