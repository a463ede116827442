"""Seeded Gaussian-mixture hidden states and random layer weights.

The paper measures on real MoE checkpoints (Mixtral-8x7B, Phi-3.5-MoE,
Qwen3-30B-A3B) and public evaluation suites; none of those are used here.
These synthetic layers stand in for them: layer shapes follow the models'
MoE blocks, hidden states follow a clustered Gaussian mixture so that
routing is sticky per sequence the way real token streams are.

Recipe (identical for every consumer):
  * numpy PCG64, root seed ``1000 + shape.index`` unless given; independent
    child streams (SeedSequence.spawn) for weights, cluster means, cluster
    draws and noise, so changing the batch or step count never changes the
    weights;
  * W_r ~ N(0, 1/d) fp32; W1, W3 ~ N(0, 1/d); W2 ~ N(0, 1/F); shared expert
    likewise with its own width; bf16 tensors are the round-to-nearest-even
    bf16 of the fp32 draw;
  * cluster means mu_c ~ N(0, 2 I_d) (variance 2); x = mu_c + N(0, I_d);
  * each sequence keeps its cluster across steps; with probability
    ``redraw`` per step it draws a new one (uniform, or Zipf(s) over
    cluster ranks when ``zipf`` is set);
  * stacked layers: layer l's weights come from root seed + 7919 l, and its
    d x d mixing matrix M_l ~ N(0, 1/d) (bf16) from a stream of its own.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
from dataclasses import dataclass, field
from typing import Optional, Tuple

import numpy as np


@dataclass(frozen=True)
class LayerShape:
    name: str
    index: int                 # 1-based position in the workload list
    d: int                     # d_model
    E: int                     # routed experts
    F: int                     # expert FFN width
    K: int                     # Top-K of the model (EAT's cap)
    top_p: Optional[float]     # Top-P threshold of the baseline, if any
    bf16: bool                 # bf16 activations and expert weights
    inv_temp: float = 1.0      # router logit scale 1/T
    F_shared: int = 0          # width of the always-on shared expert (0 = none)
    clusters: int = 4
    redraw: float = 0.1        # per-step cluster re-draw probability
    zipf: float = 0.0          # Zipf exponent for cluster popularity (0 = uniform)
    decode_batches: Tuple[int, ...] = (32,)
    decode_steps: int = 16
    prefill_tokens: int = 0
    prefill_seqs: int = 0
    layers: int = 1


SHAPES = {
    # d=128, E=8 (F=256), fp32 everywhere; 32 tokens x 16 steps, 4 clusters,
    # each token keeps its cluster for the whole run; Top-K=2, Top-P p=0.5.
    "tiny": LayerShape("tiny", 1, d=128, E=8, F=256, K=2, top_p=0.5, bf16=False,
                       clusters=4, redraw=0.0, decode_batches=(32,), decode_steps=16),
    # Mixtral-8x7B-shaped MoE block: d=4096, E=8, F=14336, bf16 experts,
    # fp32 router; logits scaled by 1/T with T=0.5; Top-K=2.
    "mixtral": LayerShape("mixtral", 2, d=4096, E=8, F=14336, K=2, top_p=None, bf16=True,
                          inv_temp=2.0, clusters=16, redraw=0.1,
                          decode_batches=(1, 8, 32, 64), decode_steps=256),
    # Fine-grained experts: d=2048, E=64, F=1024; Top-K=8, Top-P p=0.6.
    "finegrained": LayerShape("finegrained", 3, d=2048, E=64, F=1024, K=8, top_p=0.6, bf16=True,
                              clusters=32, redraw=0.1, decode_batches=(256,), decode_steps=512,
                              prefill_tokens=4096, prefill_seqs=8),
    # 60 routed experts (F=1408) + 4 shared experts fused as one F=5632 SwiGLU;
    # Zipf(1.1) cluster popularity to skew expert load; Top-K=4.
    "shared": LayerShape("shared", 4, d=2048, E=60, F=1408, K=4, top_p=None, bf16=True,
                         F_shared=5632, clusters=32, redraw=0.1, zipf=1.1,
                         decode_batches=(128,), decode_steps=256,
                         prefill_tokens=8192, prefill_seqs=16),
    # Qwen3-30B-A3B-shaped MoE block: 128 routed experts (two 64-bit mask
    # words per token), d=2048, F=768, Top-K=8; Top-P p=0.6 baseline.
    "qwen3": LayerShape("qwen3", 6, d=2048, E=128, F=768, K=8, top_p=0.6, bf16=True,
                        clusters=32, redraw=0.1, decode_batches=(64,), decode_steps=256,
                        prefill_tokens=4096, prefill_seqs=8),
    # 16 stacked finegrained layers with independent accounts.
    "stack16": LayerShape("stack16", 5, d=2048, E=64, F=1024, K=8, top_p=0.6, bf16=True,
                          clusters=64, redraw=0.1, decode_batches=(64,), decode_steps=1024,
                          layers=16),
}


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round-to-nearest-even) and return the bit
    patterns as uint16.  Used only to produce bf16 input tensors."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = u >> np.uint32(16)
    r &= np.uint32(1)
    r += np.uint32(0x7FFF)
    r += u
    r >>= np.uint32(16)
    return r.astype(np.uint16)


def _parallel(fn, jobs):
    n = min(16, os.cpu_count() or 1, max(1, len(jobs)))
    if n == 1 or sum(np.prod(j[3]) for j in jobs) < 4_000_000:
        for j in jobs:
            fn(j)
        return
    with cf.ThreadPoolExecutor(max_workers=n) as ex:
        list(ex.map(fn, jobs))


def _streams(seed: int, n: int):
    return [np.random.Generator(np.random.PCG64(s)) for s in np.random.SeedSequence(seed).spawn(n)]


def _normal(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    out = rng.standard_normal(size=shape, dtype=np.float32)
    out *= np.float32(std)
    return out


def make_layer_weights(shape: LayerShape, seed: Optional[int] = None, layer: int = 0,
                       E: Optional[int] = None, d: Optional[int] = None, F: Optional[int] = None,
                       F_shared: Optional[int] = None):
    """Return a dict of weights for one MoE layer.

    Keys: ``w_router`` fp32 [E, d]; ``w1``, ``w3`` [E, F, d]; ``w2`` [E, d, F];
    and, with a shared expert, ``ws1``, ``ws3`` [F_sh, d] and ``ws2`` [d, F_sh].
    Expert tensors are uint16 bf16 bit patterns when ``shape.bf16`` is set,
    else fp32.  ``E``/``d``/``F`` override the shape (reduced parity sizes).
    Each expert matrix is drawn from its own child stream, so a reduced E
    reuses the leading experts' values.
    """
    E = shape.E if E is None else E
    d = shape.d if d is None else d
    F = shape.F if F is None else F
    root = (1000 + shape.index if seed is None else seed) + 7919 * layer
    g_router, g_exp, g_shared = _streams(root, 3)
    w_router = _normal(g_router, (E, d), 1.0 / np.sqrt(d))
    pack = bf16_bits if shape.bf16 else (lambda a: a)
    edt = np.uint16 if shape.bf16 else np.float32
    w1 = np.empty((E, F, d), edt)
    w3 = np.empty((E, F, d), edt)
    w2 = np.empty((E, d, F), edt)
    # one child seed per (expert, matrix): values do not depend on E or on
    # how many threads draw them
    per_expert = np.random.SeedSequence(int(g_exp.integers(2**63))).spawn(max(E, shape.E))
    jobs = []
    for e in range(E):
        s1, s3, s2 = per_expert[e].spawn(3)
        jobs += [(w1, e, s1, (F, d), d), (w3, e, s3, (F, d), d), (w2, e, s2, (d, F), F)]

    def draw(job):
        dst, e, seq, shp, fan_in = job
        dst[e] = pack(_normal(np.random.Generator(np.random.PCG64(seq)), shp, 1.0 / np.sqrt(fan_in)))

    _parallel(draw, jobs)
    out = {"w_router": w_router, "w1": w1, "w3": w3, "w2": w2}
    Fs = shape.F_shared if F_shared is None else F_shared
    if Fs:
        out["ws1"] = pack(_normal(g_shared, (Fs, d), 1.0 / np.sqrt(d)))
        out["ws3"] = pack(_normal(g_shared, (Fs, d), 1.0 / np.sqrt(d)))
        out["ws2"] = pack(_normal(g_shared, (d, Fs), 1.0 / np.sqrt(Fs)))
    return out


def make_vocab_head(d: int, V: int, seed: int) -> np.ndarray:
    """A synthetic LM head W_V [V, d] ~ N(0, 1/d), bf16 bits."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(seed), 0x766f63])))
    return bf16_bits(_normal(g, (V, d), 1.0 / np.sqrt(d)))


def make_targets(S: int, V: int, seed: int) -> np.ndarray:
    """Next-token ids, uniform over the vocabulary, int32 [S]."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(seed), 0x746774])))
    return g.integers(0, V, S).astype(np.int32)


def make_expert_scale(E: int, seed: int, spread: float = 2.0) -> np.ndarray:
    """Per-expert routing scales of the kind a recovery fine-tune leaves
    behind: log-uniform in [1/spread, spread], fp32 [E]."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(seed), 0x6f7064])))
    return np.exp(g.uniform(-np.log(spread), np.log(spread), E)).astype(np.float32)


def make_mixing(shape: LayerShape, layer: int, seed: Optional[int] = None, d: Optional[int] = None) -> np.ndarray:
    """The d x d residual mixing matrix applied after stacked layer ``layer``:
    N(0, 1/d) entries from the layer's own stream, bf16 bits."""
    d = shape.d if d is None else d
    root = (1000 + shape.index if seed is None else seed) + 7919 * layer
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([root, 0x6d6978])))
    return bf16_bits(_normal(g, (d, d), 1.0 / np.sqrt(d)))


@dataclass
class HiddenStream:
    """Cluster-sticky Gaussian-mixture hidden states, one batch per step.

    ``next()`` returns x [B, d] as fp32, or as bf16 bits (uint16) when the
    shape is bf16.  ``d`` overrides the shape's width (reduced sizes).
    """
    shape: LayerShape
    batch: int
    seed: Optional[int] = None
    d: Optional[int] = None
    _state: dict = field(default_factory=dict, repr=False)

    def __post_init__(self):
        d = self.shape.d if self.d is None else self.d
        root = (1000 + self.shape.index if self.seed is None else self.seed) + 104729
        g_means, g_clusters, g_noise = _streams(root, 3)
        C = self.shape.clusters
        self._means = _normal(g_means, (C, d), np.sqrt(2.0))
        if self.shape.zipf > 0:
            w = np.arange(1, C + 1, dtype=np.float64) ** (-self.shape.zipf)
            self._pi = w / w.sum()
        else:
            self._pi = np.full(C, 1.0 / C)
        self._gc = g_clusters
        self._gn = g_noise
        self._cl = self._gc.choice(C, size=self.batch, p=self._pi)
        self._d = d
        self._first = True

    @property
    def clusters(self) -> np.ndarray:
        return self._cl.copy()

    def next(self) -> np.ndarray:
        if not self._first and self.shape.redraw > 0:
            flip = self._gc.random(self.batch) < self.shape.redraw
            nflip = int(flip.sum())
            if nflip:
                self._cl[flip] = self._gc.choice(self.shape.clusters, size=nflip, p=self._pi)
        self._first = False
        x = self._means[self._cl] + self._gn.standard_normal((self.batch, self._d), dtype=np.float32)
        x = x.astype(np.float32)
        return bf16_bits(x) if self.shape.bf16 else x

    def steps(self, n: int) -> np.ndarray:
        """Stack ``n`` consecutive steps: [n, B, d]."""
        return np.stack([self.next() for _ in range(n)])


def make_prefill(shape: LayerShape, tokens: Optional[int] = None, seqs: Optional[int] = None,
                 seed: Optional[int] = None, d: Optional[int] = None) -> np.ndarray:
    """A prefill chunk: ``seqs`` sequences laid out sequence-major, each a
    cluster-sticky run of ``tokens // seqs`` positions.  Returns [T, d]."""
    T = shape.prefill_tokens if tokens is None else tokens
    S = max(1, shape.prefill_seqs if seqs is None else seqs)
    L = T // S
    hs = HiddenStream(shape, S, seed=seed, d=d)
    x = hs.steps(L)                       # [L, S, d]
    return np.ascontiguousarray(x.transpose(1, 0, 2).reshape(S * L, -1))


def make_trend(T: int, seed: int, frac_up: float = 0.5) -> np.ndarray:
    """Per-token int8 perplexity trend in {-1, 0, +1}: +1 with probability
    ``frac_up``, else -1 or 0 with equal odds."""
    g = np.random.Generator(np.random.PCG64(seed))
    u = g.random(T)
    out = np.where(u < frac_up, 1, np.where(u < frac_up + (1 - frac_up) / 2, -1, 0))
    return out.astype(np.int8)


def make_accounts(E: int, seed: int, steps: int = 20, tokens: int = 16, c_scale: float = 1.0):
    """A plausible non-zero account state (N int64, P_total fp32, C_s fp32)
    with the shapes of the layer's state: N counts as if ``steps`` calls of
    ``tokens`` tokens had each picked a few experts; P_total a share of N;
    C_s a positive magnitude of scale ``c_scale``.  Some experts stay at 0."""
    g = np.random.Generator(np.random.PCG64(seed))
    n = g.binomial(steps * tokens, 0.2, size=E).astype(np.int64)
    n[g.random(E) < 0.2] = 0
    p = (n * g.uniform(0.1, 0.6, size=E)).astype(np.float32)
    c = np.where(n > 0, g.uniform(0.2, 1.0, size=E) * c_scale, 0.0).astype(np.float32)
    return n, p, c
