"""Plain CPU oracle of the EAT MoE-layer forward (numpy, fp64).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the test-suite, the smoke check and the CPU-baseline
leg of the benchmark use it.  It shares no code with the GPU library; the
only thing the two have in common is the seeded input arrays they are fed.

Everything is computed in float64 from the exact values of the inputs
(bf16 bit patterns are widened exactly).  The code follows the paper
("EAT: Expert Account Tracker for Efficient MoE Inference") step by step:

  Sec. 3.1  router scores -> softmax, select, renormalise, weighted sum
  Sec. 3.2  account statistics N, P_total, C_s and the history score S_h
            (Eq. 1), final importance I (Eq. 2)
  Sec. 3.3  threshold: grounding (Eq. 3-5), perplexity adjustment,
            boundedness, smoothing
  Sec. 3.4  activation set (Eq. 6), mask and renormalisation (Eq. 7-8)

Where the paper is silent or ambiguous, the readings listed in ``Params``
(and in the design notes) are applied; none is tuned per workload.

Pins: every function here is checked by ``tests/test_oracle_*.py`` against a
hand-computed three-step sequence, brute-force enumeration on E <= 8,
library routines (softmax, quantile, std, top-k, SiLU, RMSNorm, bf16
conversion) and closed forms.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

MODE_EAT, MODE_TOPK, MODE_TOPP = 0, 1, 2


@dataclass
class Params:
    """Hyper-parameters.  Defaults are the paper's table of key
    hyper-parameters (Sec. 4.1) plus the constants stated in Sec. 3.3
    (x1.2 / x0.9 perplexity factors, 10% / 90% bounds) and Eq. 7's epsilon.
    """
    mode: int = MODE_EAT
    K: int = 2                 # max activated experts (Mixtral/Phi 2, Qwen 8)
    top_p: float = 0.6         # Top-P baseline threshold
    top_p_cap: int = 0         # 0 = uncapped nucleus
    alpha: float = 0.95        # EMA factor of C_s (Sec. 3.2)
    w1: float = 0.3            # Eq. 1 weights
    w2: float = 0.3
    w3: float = 0.4
    beta: float = 0.6          # Eq. 2 balance
    alpha1: float = 0.5        # Eq. 5 scaling
    alpha2: float = 1.0
    kappa1: float = 0.7        # smoothing weights (Sec. 3.3)
    kappa2: float = 0.3
    ppl_up: float = 1.2        # perplexity rose: tau * (1 + 20%)
    ppl_down: float = 0.9      # otherwise:       tau * (1 - 10%)
    q_lo: float = 0.1          # tau_min = 10% point of the routing weights
    q_hi: float = 0.9          # tau_max = 90% point
    eps: float = 1e-8          # Eq. 7
    inv_temp: float = 1.0      # router logit scale (1 = plain softmax)
    cs_mode: int = 0           # 0: C_s used as is in Eq. 1; 1: C_s / sum(C_s)
    shared: bool = False       # always-on shared expert added with weight 1
    round_h: bool = False      # round the experts' hidden activation to bf16 (R27)
    round_y: bool = False      # round each expert's output row to bf16 before it is weighted into y,
                               # its norm still taken from the unrounded row (R27: prefill-sized calls)
    expert_scale: Optional[np.ndarray] = None   # OPD per-expert reweighting (Sec. 3.5), or None


# ---------------------------------------------------------------- inputs --

def widen(a: np.ndarray) -> np.ndarray:
    """Exact float64 view of an input tensor: uint16 arrays are bf16 bit
    patterns (the upper half of an IEEE binary32), anything else is taken
    by value."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return np.asarray(a, dtype=np.float64)       # no copy when already float64


# ------------------------------------------------------- router (Sec 3.1) --

def router_probs(x: np.ndarray, w_router: np.ndarray, inv_temp: float = 1.0) -> np.ndarray:
    """Router scores z = x W_r^T (scaled by 1/T) and their softmax over all
    experts, row by row (Sec. 3.1; p_i of Eq. 2 and g_i of Eq. 3-7 are this
    same probability vector)."""
    z = widen(x) @ widen(w_router).T * inv_temp
    z = z - z.max(axis=1, keepdims=True)
    ez = np.exp(z)
    return ez / ez.sum(axis=1, keepdims=True)


# ----------------------------------------------- history score (Sec 3.2) --

def history_score(n: np.ndarray, p_total: np.ndarray, c_s: np.ndarray, prm: Params) -> np.ndarray:
    """Eq. 1:  S_h,i = w1 N_i / sum N + w2 P_total,i / N_i + w3 C_s,i.

    0/0 reads as 0: the first term is 0 while no expert has been activated,
    the second is 0 for an expert never activated.  With ``cs_mode`` 1 the
    third term uses C_s,i / sum C_s (0 while all C_s are 0)."""
    E = len(n)
    n = np.asarray(n, dtype=np.int64)
    total = int(n.sum())
    s = np.zeros(E)
    csum = float(np.sum(np.asarray(c_s, dtype=np.float64)))
    for i in range(E):
        t1 = n[i] / total if total > 0 else 0.0
        t2 = float(p_total[i]) / n[i] if n[i] > 0 else 0.0
        if prm.cs_mode == 0:
            t3 = float(c_s[i])
        else:
            t3 = float(c_s[i]) / csum if csum > 0 else 0.0
        s[i] = prm.w1 * t1 + prm.w2 * t2 + prm.w3 * t3
    return s


def importance(p_row: np.ndarray, s_h: np.ndarray, beta: float) -> np.ndarray:
    """Eq. 2:  I_i = (1 - beta) p_i + beta S_h,i."""
    return (1.0 - beta) * p_row + beta * s_h


# -------------------------------------------------- threshold (Sec 3.3) --

def grounding(g_row: np.ndarray, alpha1: float, alpha2: float):
    """Eq. 3-5: mean mu_w and population standard deviation sigma_w of the
    gating scores, tau = max(alpha1 mu_w, mu_w - alpha2 sigma_w)."""
    E = len(g_row)
    mu = sum(float(v) for v in g_row) / E
    var = sum((float(v) - mu) ** 2 for v in g_row) / E
    sigma = math.sqrt(var)
    return mu, sigma, max(alpha1 * mu, mu - alpha2 * sigma)


def quantile(values: np.ndarray, q: float) -> float:
    """The q-point of a row of routing weights: sort ascending, position
    h = q (E - 1), interpolate linearly between its two neighbours."""
    v = sorted(float(a) for a in values)
    h = q * (len(v) - 1)
    lo = int(math.floor(h))
    hi = min(lo + 1, len(v) - 1)
    return v[lo] + (h - lo) * (v[hi] - v[lo])


def threshold(g_row: np.ndarray, trend: int, prm: Params) -> dict:
    """Sec. 3.3 end to end for one token.

    * grounding tau (Eq. 3-5);
    * perplexity adjustment: tau_PPL = 1.2 tau when the perplexity trend is
      positive, else 0.9 tau (no signal counts as "otherwise");
    * smoothing: kappa1 tau_PPL + kappa2 tau (mixes with the current tau);
    * bounds: the smoothed value is clamped to [tau_min, tau_max], the 10%
      and 90% points of this token's routing weights; the clamp is applied
      last so that the stated bound holds for tau_final.
    """
    mu, sigma, tau = grounding(g_row, prm.alpha1, prm.alpha2)
    f = prm.ppl_up if trend > 0 else prm.ppl_down
    tau_ppl = f * tau
    tau_s = prm.kappa1 * tau_ppl + prm.kappa2 * tau
    t_min = quantile(g_row, prm.q_lo)
    t_max = quantile(g_row, prm.q_hi)
    tau_final = min(max(tau_s, t_min), t_max)
    return dict(mu=mu, sigma=sigma, tau=tau, tau_ppl=tau_ppl, tau_s=tau_s,
                tau_min=t_min, tau_max=t_max, tau_final=tau_final)


# -------------------------------------------------- selection (Sec 3.4) --

def select_eat(I: np.ndarray, tau_final: float, K: int) -> List[int]:
    """Eq. 6.  Candidates are the experts with I_i > tau_final (strict).
    None: the single arg-max of I (lowest index on a tie).  Up to K: all of
    them.  More than K: every candidate that fewer than K other candidates
    strictly beat (so exact ties at the K-th value are all kept)."""
    E = len(I)
    cand = [i for i in range(E) if I[i] > tau_final]
    if len(cand) == 0:
        best = 0
        for i in range(1, E):
            if I[i] > I[best]:
                best = i
        return [best]
    if len(cand) <= K:
        return cand
    out = []
    for i in cand:
        beaten_by = sum(1 for j in cand if I[j] > I[i])
        if beaten_by < K:
            out.append(i)
    return out


def _descending_order(p: np.ndarray) -> List[int]:
    # Largest first; equal values keep the lower expert index first.
    return sorted(range(len(p)), key=lambda i: (-float(p[i]), i))


def select_topk(p_row: np.ndarray, K: int) -> List[int]:
    """Vanilla Top-K routing (Sec. 3.1): the K largest routing
    probabilities; ties go to the lower expert index."""
    return sorted(_descending_order(p_row)[:K])


def select_topp(p_row: np.ndarray, p_thr: float, cap: int = 0) -> List[int]:
    """Top-P routing (the dynamic baseline of Sec. 4.1): walk the
    probabilities from the largest down and stop at the first prefix whose
    sum reaches p_thr.  ``cap`` > 0 limits the prefix length."""
    chosen, acc = [], 0.0
    for i in _descending_order(p_row):
        chosen.append(i)
        acc += float(p_row[i])
        if acc >= p_thr:
            break
        if cap and len(chosen) >= cap:
            break
    return sorted(chosen)


def renormalise(g_row: np.ndarray, sel: Sequence[int], eps: float) -> np.ndarray:
    """Eq. 7-8: m_i = 1 for selected experts, g_norm,i = g_i m_i /
    (sum_j g_j m_j + eps)."""
    m = np.zeros(len(g_row))
    m[list(sel)] = 1.0
    num = g_row * m
    return num / (num.sum() + eps)


def mask_of(sel: Sequence[int]) -> int:
    out = 0
    for i in sel:
        out |= 1 << int(i)
    return out


# ------------------------------------------------------------ routing ---

@dataclass
class Routing:
    p: np.ndarray              # [T, E] router probabilities
    masks: List[int]           # bit i set <=> expert i selected
    k: np.ndarray              # [T] number selected
    g_norm: np.ndarray         # [T, E] renormalised gates (0 off-mask)
    I: Optional[np.ndarray] = None          # [T, E] (EAT only)
    s_h: Optional[np.ndarray] = None        # [E]    (EAT only)
    thr: List[dict] = field(default_factory=list)   # per-token Sec. 3.3 values

    def selected(self, t: int) -> List[int]:
        m = self.masks[t]
        return [i for i in range(self.p.shape[1]) if (m >> i) & 1]


def reweight(p: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """Sec. 3.5 (OPD at inference): scale each expert's raw routing
    probability and renormalise the row, p'_i = s_i p_i / sum_j s_j p_j."""
    q = np.asarray(p, dtype=np.float64) * widen(scale)[None, :]
    return q / q.sum(axis=1, keepdims=True)


def route_probs(p: np.ndarray, acc, trend: Optional[np.ndarray], prm: Params) -> Routing:
    """Selection and renormalisation for a block of tokens whose router
    probabilities are already known.  Every token is judged against the
    same account snapshot ``acc`` = (N, P_total, C_s).  With an OPD scale
    the reweighted probabilities take the place of p everywhere below."""
    p = np.asarray(p, dtype=np.float64)
    if prm.expert_scale is not None:
        p = reweight(p, prm.expert_scale)
    T, E = p.shape
    masks, ks = [], np.zeros(T, dtype=np.int64)
    g = np.zeros((T, E))
    I_all = np.zeros((T, E)) if prm.mode == MODE_EAT else None
    s_h = history_score(acc[0], acc[1], acc[2], prm) if prm.mode == MODE_EAT else None
    thr = []
    for t in range(T):
        row = p[t]
        if prm.mode == MODE_TOPK:
            sel = select_topk(row, prm.K)
        elif prm.mode == MODE_TOPP:
            sel = select_topp(row, prm.top_p, prm.top_p_cap)
        else:
            tr = 0 if trend is None else int(trend[t])
            th = threshold(row, tr, prm)
            I = importance(row, s_h, prm.beta)
            I_all[t] = I
            sel = select_eat(I, th["tau_final"], prm.K)
            thr.append(th)
        masks.append(mask_of(sel))
        ks[t] = len(sel)
        g[t] = renormalise(row, sel, prm.eps)
    return Routing(p=p, masks=masks, k=ks, g_norm=g, I=I_all, s_h=s_h, thr=thr)


def route(x, w_router, acc, trend, prm: Params) -> Routing:
    return route_probs(router_probs(x, w_router, prm.inv_temp), acc, trend, prm)


# ------------------------------------------------------------ experts ---

def silu(a: np.ndarray) -> np.ndarray:
    return a / (1.0 + np.exp(-a))


def swiglu(x: np.ndarray, w1: np.ndarray, w3: np.ndarray, w2: np.ndarray, round_h: bool = False) -> np.ndarray:
    """One expert FFN applied to rows of x: W2 (silu(W1 x) * (W3 x)), no
    biases.  x [n, d]; w1, w3 [F, d]; w2 [d, F]; returns [n, d].  With
    ``round_h`` the hidden activation is rounded to bf16 before W2, the
    precision at which a bf16 layer stores it (reading R27)."""
    x = widen(x)
    h = silu(x @ widen(w1).T) * (x @ widen(w3).T)
    if round_h:
        h = round_bf16(h)
    return h @ widen(w2).T


@dataclass
class LayerOut:
    y: np.ndarray              # [T, d] (rows outside ``tokens`` are 0)
    norms: np.ndarray          # [T, E] ||o_{t,e}||_2 of un-gated outputs (0 off-mask)


def layer_outputs(x, weights: dict, r: Routing, prm: Params, tokens: Optional[Sequence[int]] = None) -> LayerOut:
    """Sec. 3.1 / Eq. 7-8: y_t = sum_{e selected} g_norm,t,e Expert_e(x_t),
    plus the always-on shared expert with weight 1 when present.  Only the
    rows in ``tokens`` are computed (all by default).  With ``round_y`` each
    expert's output row enters y rounded to bf16 (its norm does not)."""
    T, E = r.p.shape
    toks = list(range(T)) if tokens is None else sorted(set(int(t) for t in tokens))
    xw = widen(x)
    d = xw.shape[1]
    y = np.zeros((T, d))
    norms = np.zeros((T, E))
    for e in range(E):
        rows = [t for t in toks if (r.masks[t] >> e) & 1]
        if not rows:
            continue
        o = swiglu(xw[rows], weights["w1"][e], weights["w3"][e], weights["w2"][e], prm.round_h)
        for j, t in enumerate(rows):
            norms[t, e] = math.sqrt(float(np.dot(o[j], o[j])))
            y[t] += r.g_norm[t, e] * (round_bf16(o[j]) if prm.round_y else o[j])
    if prm.shared and "ws1" in weights:
        o = swiglu(xw[toks], weights["ws1"], weights["ws3"], weights["ws2"], prm.round_h)
        for j, t in enumerate(toks):
            y[t] += o[j]
    return LayerOut(y=y, norms=norms)


# ----------------------------------------------- account update (Sec 3.2) --

def account_update(acc, r_masks: Sequence[int], p: np.ndarray, norms: np.ndarray, prm: Params):
    """Sec. 3.2 bookkeeping after one forward step.

    For each expert i activated by n_i > 0 tokens of the step:
      N_i       += n_i                       (activation count)
      P_total,i += sum of those tokens' p_i  (router weight collected)
      C_s,i      = (1 - alpha) C_s,i + alpha * mean of their ||o||_2
    Experts not activated keep their values.  Sums are exact-rounded in
    float64 (math.fsum) and rounded once to the float32 state.
    """
    n_in, p_in, c_in = acc
    E = len(n_in)
    n_out = np.array(n_in, dtype=np.int64).copy()
    p_out = np.array(p_in, dtype=np.float32).copy()
    c_out = np.array(c_in, dtype=np.float32).copy()
    for i in range(E):
        toks = [t for t, m in enumerate(r_masks) if (m >> i) & 1]
        if not toks:
            continue
        n_out[i] += len(toks)
        p_out[i] = np.float32(math.fsum([float(p_in[i])] + [float(p[t, i]) for t in toks]))
        mean_norm = math.fsum(float(norms[t, i]) for t in toks) / len(toks)
        c_out[i] = np.float32((1.0 - prm.alpha) * float(c_in[i]) + prm.alpha * mean_norm)
    return n_out, p_out, c_out


def zero_accounts(E: int):
    return np.zeros(E, np.int64), np.zeros(E, np.float32), np.zeros(E, np.float32)


# --------------------------------------------------------- whole step ---

@dataclass
class StepOut:
    y: np.ndarray
    routing: Routing
    norms: np.ndarray
    acc: tuple


def moe_step(x, weights: dict, acc, trend, prm: Params, sequential: bool = False) -> StepOut:
    """One MoE-layer forward over a block of tokens.

    Default (snapshot): every token routes against the accounts as they are
    at the start of the step; one aggregated account update follows (EAT
    mode only).  ``sequential=True`` routes and accounts one token at a
    time in order; at one token per step both agree."""
    if sequential:
        T = widen(x).shape[0]
        ys, ms, ps, gs, ns, ks, Is, ths = [], [], [], [], [], [], [], []
        cur = acc
        for t in range(T):
            tr = None if trend is None else np.asarray(trend)[t:t + 1]
            o = moe_step(np.asarray(x)[t:t + 1], weights, cur, tr, prm, sequential=False)
            ys.append(o.y[0]); ms.append(o.routing.masks[0]); ps.append(o.routing.p[0])
            gs.append(o.routing.g_norm[0]); ns.append(o.norms[0]); ks.append(o.routing.k[0])
            ths += o.routing.thr
            if o.routing.I is not None:
                Is.append(o.routing.I[0])
            cur = o.acc
        r = Routing(p=np.array(ps), masks=ms, k=np.array(ks), g_norm=np.array(gs),
                    I=np.array(Is) if Is else None, thr=ths)
        return StepOut(y=np.array(ys), routing=r, norms=np.array(ns), acc=cur)
    r = route(x, weights["w_router"], acc, trend, prm)
    lo = layer_outputs(x, weights, r, prm)
    new_acc = account_update(acc, r.masks, r.p, lo.norms, prm) if prm.mode == MODE_EAT else acc
    return StepOut(y=lo.y, routing=r, norms=lo.norms, acc=new_acc)


# ------------------------------------------- stacked layers (evaluation) --
#
# The 16-layer evaluation workload composes MoE layers, each with its own
# account state: layer l reads u = RMSNorm(h_l) (unit weight), and the next
# layer's input is h_{l+1} = (h_l + MoE_l(u)) M_l^T with a d x d mixing
# matrix.  Activations are bf16 between the steps, rounded once at each of
# the three points below from the exact (here fp64) value.

def round_bf16(a) -> np.ndarray:
    """Nearest bf16 value (ties to even) of each element, as float64:
    8 significant bits, quantum 2**(e - 8) for a value in [2**(e-1), 2**e),
    never finer than the smallest subnormal step 2**-133."""
    a = np.asarray(a, dtype=np.float64)
    _, e = np.frexp(a)
    q = np.ldexp(1.0, np.maximum(e, -125) - 8)
    out = np.rint(a / q) * q                       # rint rounds halves to even
    return np.where(np.abs(out) > 3.3895313892515355e38, np.copysign(np.inf, a), out)


def rms_norm(h, eps: float = 1e-6) -> np.ndarray:
    """Row-wise h / sqrt(mean(h^2) + eps) (unit gain)."""
    h = widen(h)
    return h / np.sqrt(np.mean(h * h, axis=1, keepdims=True) + eps)


@dataclass
class StackOut:
    h: np.ndarray              # [T, d] bf16 values (float64) after the last layer
    layers: List[StepOut]      # per layer: routing, outputs, new accounts


def stack_step(x, layers: Sequence[dict], mixes: Sequence[np.ndarray], accs: Sequence[tuple], trend,
               prms: Sequence[Params], eps: float = 1e-6) -> StackOut:
    """One decode step through the stacked layers:
    u_l = bf16(RMSNorm(h_l)), r_l = bf16(h_l + MoE_l(u_l)), h_{l+1} = bf16(r_l M_l^T)."""
    h = widen(x)
    outs = []
    for w, m, acc, prm in zip(layers, mixes, accs, prms):
        u = round_bf16(rms_norm(h, eps))
        o = moe_step(u, w, acc, trend, prm)
        r = round_bf16(h + o.y)
        h = round_bf16(r @ widen(m).T)
        outs.append(o)
    return StackOut(h=h, layers=outs)


# ------------------------------------------- perplexity signal (Sec 3.3) --
#
# The threshold's performance-based adjustment compares the current model
# perplexity with the previous one.  Per sequence: the token's negative
# log-likelihood under the LM head, NLL = logsumexp(h W_V^T) - (h W_V^T)[y],
# a running perplexity exp(sum NLL / n) over the sequence so far, and the
# trend +1 when it rose since the sequence's previous token, -1 when it did
# not, 0 for a sequence's first token (reading R30).

@dataclass
class PplState:
    nll_sum: np.ndarray        # [S] float64
    count: np.ndarray          # [S] int64
    ppl_prev: np.ndarray       # [S] float64


def ppl_zero_state(S: int) -> PplState:
    return PplState(np.zeros(S), np.zeros(S, np.int64), np.zeros(S))


def ppl_update(h, w_vocab, target, state: PplState):
    """One token per sequence: returns (nll [S], ppl [S], trend [S] int8,
    new state)."""
    z = widen(h) @ widen(w_vocab).T
    zmax = z.max(axis=1, keepdims=True)
    lse = zmax[:, 0] + np.log(np.exp(z - zmax).sum(axis=1))
    tgt = np.asarray(target, dtype=np.int64)
    nll = lse - z[np.arange(z.shape[0]), tgt]
    nll_sum = state.nll_sum + nll
    count = state.count + 1
    ppl = np.exp(nll_sum / count)
    trend = np.where(count > 1, np.where(ppl > state.ppl_prev, 1, -1), 0).astype(np.int8)
    return nll, ppl, trend, PplState(nll_sum, count, ppl)
