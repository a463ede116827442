"""Comparison helpers for GPU-vs-oracle parity tests.

A token is *borderline* when its selection is decided by a margin smaller
than the arithmetic can resolve: the GPU routes in fp32, the oracle in
fp64, so a score within eps_b of the threshold (or of the K-th / (K+1)-th
rank, or of the Top-P threshold) may legitimately fall either way.  The
decision is taken on the oracle's values only.  Masks of all other tokens
must match bit for bit; borderline tokens are counted and reported.
"""
from __future__ import annotations

import numpy as np

import oracle as O

EPS_B = 1e-6          # least borderline band (scaled by max(1, max|I|) in EAT mode)
BAND_MAX = 1e-5       # a call whose observed |dp| asks for a wider band fails
TOL_Y_F32 = 1e-4      # per-token max|dy| / max|y| for fp32 layers
TOL_Y_BF16 = 2e-2     # same for bf16 experts (H rounded to bf16, y stored as bf16)
TOL_P = 2e-5          # |p_gpu - p_oracle| and gate differences
TOL_C_F32 = 1e-5      # relative, C_s after a step
TOL_C_BF16 = 1e-2
TOL_P_TOTAL = 1e-5


def borderline(r: O.Routing, prm: O.Params, eps_b=EPS_B, shift=0.0) -> np.ndarray:
    """Tokens whose selection the oracle's values decide within the band
    ``eps_b`` (a scalar, or one band per token).  In EAT mode the band is
    relative (scaled by max(1, max|I|)) and ``shift`` (scalar or per token)
    adds an absolute bound on the importance difference that comes from the
    two sides' account states differing (Eq. 1-2)."""
    T, E = r.p.shape
    out = np.zeros(T, dtype=bool)
    bands = np.broadcast_to(np.asarray(eps_b, dtype=np.float64), (T,))
    shifts = np.broadcast_to(np.asarray(shift, dtype=np.float64), (T,))
    for t in range(T):
        eps_b = float(bands[t])
        p = r.p[t]
        if prm.mode == O.MODE_EAT:
            I = r.I[t]
            tf = r.thr[t]["tau_final"]
            eb = eps_b * max(1.0, float(np.abs(I).max())) + float(shifts[t])
            if np.any(np.abs(I - tf) <= eb):
                out[t] = True
                continue
            cand = np.sort(I[I > tf])[::-1]
            if len(cand) > prm.K and cand[prm.K - 1] - cand[prm.K] <= eb:
                out[t] = True
            if len(cand) == 0:
                srt = np.sort(I)[::-1]
                if E > 1 and srt[0] - srt[1] <= eb:
                    out[t] = True
        elif prm.mode == O.MODE_TOPK:
            srt = np.sort(p)[::-1]
            if prm.K < E and srt[prm.K - 1] - srt[prm.K] <= eps_b:
                out[t] = True
        else:
            srt = np.sort(p)[::-1]
            c = np.cumsum(srt)
            k = int(r.k[t])
            if abs(c[k - 1] - prm.top_p) <= eps_b or (k >= 2 and abs(c[k - 2] - prm.top_p) <= eps_b):
                out[t] = True
            if np.any(np.abs(np.diff(srt[:k + 1])) <= eps_b):   # order of near-equal values
                out[t] = True
    return out


def masks_to_list(mask_tensor) -> list:
    """[T] or [T, W] uint64 words (word j holds experts 64 j .. 64 j + 63)
    -> one Python int per token, bit e <=> expert e."""
    a = mask_tensor.detach().cpu().numpy().astype(np.int64).view(np.uint64)
    if a.ndim == 1:
        return [int(v) for v in a]
    return [sum(int(w) << (64 * j) for j, w in enumerate(row)) for row in a]


def row_rel_err(y_gpu: np.ndarray, y_ref: np.ndarray) -> np.ndarray:
    den = np.maximum(np.abs(y_ref).max(axis=1), 1e-30)
    return np.abs(y_gpu - y_ref).max(axis=1) / den


def oracle_params(shape, mode: int, K=None, top_p=None, cs_mode: int = 0, shared: bool = False) -> O.Params:
    return O.Params(mode=mode, K=shape.K if K is None else K,
                    top_p=(shape.top_p or 0.6) if top_p is None else top_p,
                    inv_temp=shape.inv_temp, cs_mode=cs_mode, shared=shared)


def report(name: str, **kv) -> None:
    items = " ".join(f"{k}={v}" for k, v in kv.items())
    print(f"[parity] {name}: {items}", flush=True)


def band_for(dp: float) -> float:
    """Borderline band of a call: 4x the largest router-probability
    difference observed between the two sides (|dI| <= (1 - beta) |dp| plus
    the fp32 rounding of S_h, which the max(1, max|I|) scale covers), never
    below EPS_B.  A wider band than BAND_MAX means the probabilities
    themselves disagree, which the caller reports as a failure."""
    return max(EPS_B, 4.0 * float(dp))


def _bits(m: int, E: int) -> np.ndarray:
    return np.array([(m >> e) & 1 for e in range(E)], dtype=bool)


def valid_choice(m: int, r: O.Routing, t: int, prm: O.Params, band: float, shift: float = 0.0) -> str:
    """Is mask ``m`` a correct selection for token t of routing ``r`` when
    every value the decision compares may be off by ``band``?  Returns "" if
    it is, else the rule it breaks.

    EAT (Eq. 6), with eb = band * max(1, max|I|) + shift: "sure" candidates have
    I > tau_final + eb, "possible" ones I > tau_final - eb.  The mask must be
    one of the three outcomes of Eq. 6 for some candidate set between the
    two: the argmax of I (no sure candidate; its I within eb of the largest),
    the whole candidate set (at most K experts, every sure one included, none
    outside the possible ones), or the rank-capped set (at least K possible
    candidates, each beaten by fewer than K possible candidates by more than
    eb, and every sure candidate left out beaten by at least K selected ones
    to within eb).
    Top-K: exactly K experts, none outweighed by an unselected one by more
    than the band.  Top-P: a descending prefix to within the band whose sum
    reaches p (or that stops at the cap) and that would not have stopped one
    expert earlier."""
    E = r.p.shape[1]
    sel = _bits(m, E)
    if not sel.any():
        return "no expert selected"
    p = r.p[t]
    if prm.mode == O.MODE_EAT:
        I = r.I[t]
        tf = r.thr[t]["tau_final"]
        eb = band * max(1.0, float(np.abs(I).max())) + shift
        sure, maybe = I > tf + eb, I > tf - eb
        n = int(sel.sum())
        if n == 1 and not sure.any() and I[sel][0] >= I.max() - eb:
            return ""                                           # argmax of I
        if n <= prm.K and not (sure & ~sel).any() and not (sel & ~maybe).any():
            return ""                                           # the candidate set
        if n >= prm.K and not (sel & ~maybe).any():
            Im = I[maybe]
            if all(int((Im > I[s] + eb).sum()) < prm.K for s in np.flatnonzero(sel)) and \
               all(int((I[sel] > I[u] - eb).sum()) >= prm.K for u in np.flatnonzero(sure & ~sel)):
                return ""                                       # rank-capped (Eq. 6, |E| > K)
        return "no outcome of Eq. 6 within the band"
    if (~sel).any() and p[sel].min() < p[~sel].max() - band:
        return "an unselected expert outweighs a selected one"
    if prm.mode == O.MODE_TOPK:
        return "" if int(sel.sum()) == prm.K else "not K experts"
    k = int(sel.sum())
    if prm.top_p_cap and k > prm.top_p_cap:
        return "more experts than the cap"
    at_cap = bool(prm.top_p_cap) and k == prm.top_p_cap
    if not at_cap and p[sel].sum() < prm.top_p - band:
        return "the prefix does not reach p"
    if k > 1 and p[sel].sum() - p[sel].min() >= prm.top_p + band:
        return "the prefix reached p one expert earlier"
    return ""


def adopt(r: O.Routing, gm, border: np.ndarray, prm: O.Params) -> O.Routing:
    """The oracle's routing with each borderline token's selection replaced by
    the GPU's (after ``valid_choice`` accepted it) and its gates renormalised
    from the oracle's own probabilities (Eq. 7-8): the several correct
    answers of a borderline token are thereby narrowed to the one the GPU
    took, and the layer output and account update that follow from it are
    still the oracle's.  Non-borderline tokens keep the oracle's masks."""
    masks = list(r.masks)
    k = r.k.copy()
    g = r.g_norm.copy()
    for t in np.flatnonzero(border):
        masks[t] = int(gm[t])
        sel = [e for e in range(r.p.shape[1]) if (masks[t] >> e) & 1]
        k[t] = len(sel)
        g[t] = O.renormalise(r.p[t], sel, prm.eps)
    return O.Routing(p=r.p, masks=masks, k=k, g_norm=g, I=r.I, s_h=r.s_h, thr=r.thr)


def compare_masks(name: str, gm, r: O.Routing, prm: O.Params, band, shift=0.0) -> tuple:
    """Masks of every token: bit-exact where the oracle's values decide the
    selection by more than the band, a valid selection (``valid_choice``)
    where they do not.  Returns (borderline flags, the routing with the GPU's
    borderline choices adopted).  ``band`` and ``shift`` (see ``borderline``)
    are scalars or one per token."""
    T = len(gm)
    bands = np.broadcast_to(np.asarray(band, dtype=np.float64), (T,))
    shifts = np.broadcast_to(np.asarray(shift, dtype=np.float64), (T,))
    border = borderline(r, prm, eps_b=bands, shift=shifts)
    bad = [t for t in range(T) if not border[t] and gm[t] != r.masks[t]]
    assert not bad, f"{name}: {len(bad)} mask mismatches outside the band, e.g. token {bad[0]}"
    for t in np.flatnonzero(border):
        why = valid_choice(gm[t], r, t, prm, float(bands[t]), float(shifts[t]))
        assert not why, f"{name}: borderline token {t}: {why}"
    return border, adopt(r, gm, border, prm)


def history_shift(acc_gpu, acc_ref, prm: O.Params) -> float:
    """Bound on the importance difference (Eq. 2) that two account states
    cause: beta times the largest difference of their history scores (Eq. 1),
    doubled for margin.  Used as the absolute ``shift`` of the band when the
    GPU routes against its own accounts and the oracle against its own."""
    if prm.mode != O.MODE_EAT:
        return 0.0
    a = O.history_score(*acc_gpu, prm)
    b = O.history_score(*acc_ref, prm)
    return 2.0 * prm.beta * float(np.abs(a - b).max())


class CachedWeights(dict):
    """A layer's weights with each expert matrix widened to float64 once and
    kept (the oracle widens per call; full-size tests reuse an expert across
    steps).  Indexing ``w["w1"][e]`` returns the cached float64 matrix."""

    class _Experts:
        def __init__(self, a):
            self.a, self.c = a, {}

        def __getitem__(self, e):
            if e not in self.c:
                self.c[e] = O.widen(self.a[e])
            return self.c[e]

        def __len__(self):
            return len(self.a)

    def __init__(self, w):
        super().__init__(w)
        for k in ("w1", "w3", "w2"):
            self[k] = CachedWeights._Experts(w[k])
        for k in ("ws1", "ws3", "ws2"):
            if k in w:
                self[k] = O.widen(w[k])


def rows_bf16(T: int, K: int, E: int, d: int, F: int) -> bool:
    """Whether a bf16 layer call of T tokens takes the library's prefill-sized
    path, whose down projection stores the expert rows in bf16 once their
    norms are taken (reading R27): T K >= 256 E rows, with the wide tiles'
    shapes (F a multiple of 128, d of 256)."""
    return T * K >= 256 * E and F % 128 == 0 and d % 256 == 0


def stack_follow(x, layers, mixes, accs, prms, pick, eps: float = 1e-6) -> O.StackOut:
    """The oracle's stacked-layer step, composed here from its pinned parts
    exactly as ``O.stack_step`` composes them (u = bf16(RMSNorm(h)),
    r = bf16(h + MoE(u)), h' = bf16(r M^T)), with a hook between each layer's
    routing and its experts: ``pick(l, routing)`` returns the routing to use
    -- the oracle's with the GPU's validated borderline choices adopted, so
    the two sides stay on one path through all layers.  With ``pick``
    returning its argument this is ``O.stack_step`` (tested on the CPU)."""
    h = O.widen(x)
    outs = []
    for l, (w, m, acc, prm) in enumerate(zip(layers, mixes, accs, prms)):
        u = O.round_bf16(O.rms_norm(h, eps))
        r = pick(l, O.route(u, w["w_router"], acc, None, prm))
        lo = O.layer_outputs(u, w, r, prm)
        new_acc = O.account_update(acc, r.masks, r.p, lo.norms, prm) if prm.mode == O.MODE_EAT else acc
        res = O.round_bf16(h + lo.y)
        h = O.round_bf16(res @ O.widen(m).T)
        outs.append(O.StepOut(y=lo.y, routing=r, norms=lo.norms, acc=new_acc))
    return O.StackOut(h=h, layers=outs)
