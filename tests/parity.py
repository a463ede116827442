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

EPS_B = 1e-5          # borderline band (scaled by max(1, max|I|) in EAT mode)
TOL_Y_F32 = 1e-4      # per-token max|dy| / max|y| for fp32 layers
TOL_Y_BF16 = 2e-2     # same for bf16 experts (H rounded to bf16, y stored as bf16)
TOL_P = 2e-5          # |p_gpu - p_oracle| and gate differences
TOL_C_F32 = 1e-5      # relative, C_s after a step
TOL_C_BF16 = 1e-2
TOL_P_TOTAL = 1e-5


def borderline(r: O.Routing, prm: O.Params, eps_b=EPS_B) -> np.ndarray:
    """Tokens whose selection the oracle's values decide within the band
    ``eps_b`` (a scalar, or one band per token)."""
    T, E = r.p.shape
    out = np.zeros(T, dtype=bool)
    bands = np.broadcast_to(np.asarray(eps_b, dtype=np.float64), (T,))
    for t in range(T):
        eps_b = float(bands[t])
        p = r.p[t]
        if prm.mode == O.MODE_EAT:
            I = r.I[t]
            tf = r.thr[t]["tau_final"]
            eb = eps_b * max(1.0, float(np.abs(I).max()))
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
