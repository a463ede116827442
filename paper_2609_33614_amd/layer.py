"""A small owner object around one EAT layer handle.

Holds the handle, the caller-owned account tensors and a workspace
allocated with torch (device memory plumbing only), and forwards to the C
entry points of ``_lib``.  All compute runs in libeat.so.
"""
from __future__ import annotations

from typing import Dict, Optional

import torch

from . import _lib as L


class EatLayer:
    def __init__(self, params: L.eat_params_t, max_tokens: int, weights: Dict[str, torch.Tensor],
                 device: str = "cuda"):
        self.params = params
        self.max_tokens = int(max_tokens)
        self.device = torch.device(device)
        self.handle = L.eat_create(params, max_tokens)
        self.w = weights
        E = params.E
        self.n = torch.zeros(E, dtype=torch.int64, device=self.device)
        self.p_total = torch.zeros(E, dtype=torch.float32, device=self.device)
        self.c_s = torch.zeros(E, dtype=torch.float32, device=self.device)
        self._ws: Optional[torch.Tensor] = None

    # account state -------------------------------------------------------
    @property
    def acc(self) -> L.eat_accounts_t:
        return L.accounts(self.n, self.p_total, self.c_s)

    def reset_accounts(self, stream=None) -> None:
        L.eat_reset_accounts(self.handle, self.acc, stream)

    def load_accounts(self, n, p_total, c_s) -> None:
        self.n.copy_(torch.as_tensor(n, dtype=torch.int64))
        self.p_total.copy_(torch.as_tensor(p_total, dtype=torch.float32))
        self.c_s.copy_(torch.as_tensor(c_s, dtype=torch.float32))

    def accounts_host(self):
        return (self.n.cpu().numpy(), self.p_total.cpu().numpy(), self.c_s.cpu().numpy())

    # workspace -----------------------------------------------------------
    def workspace(self, T: int) -> torch.Tensor:
        need = L.eat_workspace_size(self.handle, T)
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        return self._ws

    # calls ---------------------------------------------------------------
    def forward(self, x: torch.Tensor, trend: Optional[torch.Tensor] = None, y: Optional[torch.Tensor] = None,
                mask_out: Optional[torch.Tensor] = None, load_out: Optional[torch.Tensor] = None,
                stream=None, events=None) -> torch.Tensor:
        T = x.shape[0]
        if y is None:
            y = torch.empty_like(x)
        ws = self.workspace(T)
        w = self.w
        args = (self.handle, x, T, w["w_router"], w["w1"], w["w3"], w["w2"], w.get("ws1"), w.get("ws3"),
                w.get("ws2"), self.acc, trend, y, mask_out, load_out, ws, ws.numel(), stream)
        if events is None:
            L.eat_moe_forward(*args)
        else:
            L.eat_moe_forward_profiled(*args, events=events)
        return y

    def mask_tensor(self, T: int) -> torch.Tensor:
        """Mask output for T tokens: [T] for E <= 64, else [T, words]."""
        W = L.mask_words(self.params.E)
        return torch.empty((T,) if W == 1 else (T, W), dtype=torch.int64, device=self.device)

    def route(self, x: torch.Tensor, trend: Optional[torch.Tensor] = None, stream=None):
        T = x.shape[0]
        E = self.params.E
        mask = self.mask_tensor(T)
        k = torch.empty(T, dtype=torch.int32, device=self.device)
        gate = torch.empty(T, E, dtype=torch.float32, device=self.device)
        prob = torch.empty(T, E, dtype=torch.float32, device=self.device)
        ws = self.workspace(T)
        L.eat_route(self.handle, x, T, self.w["w_router"], self.acc, trend, mask, k, gate, prob,
                    ws, ws.numel(), stream)
        return mask, k, gate, prob

    def close(self) -> None:
        if self.handle:
            L.eat_destroy(self.handle)
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class PplSignal:
    """Running perplexity of S sequences through an LM head (Sec. 3.3's
    signal): ``step(h, target)`` returns the int8 trend for the sequences'
    next tokens (eat_ppl_trend)."""

    def __init__(self, S: int, w_vocab: torch.Tensor, device: str = "cuda"):
        self.S, self.w = int(S), w_vocab
        self.V, self.d = w_vocab.shape
        dev = torch.device(device)
        self.nll_sum = torch.zeros(S, dtype=torch.float64, device=dev)
        self.count = torch.zeros(S, dtype=torch.int32, device=dev)
        self.ppl_prev = torch.zeros(S, dtype=torch.float64, device=dev)
        self.trend = torch.zeros(S, dtype=torch.int8, device=dev)
        self.nll = torch.zeros(S, dtype=torch.float32, device=dev)
        self.ws = torch.empty(max(256, L.eat_ppl_workspace_size(S, self.d, self.V)), dtype=torch.uint8, device=dev)

    def reset(self, stream=None) -> None:
        L.eat_ppl_reset(self.S, self.nll_sum, self.count, self.ppl_prev, stream)

    def step(self, h: torch.Tensor, target: torch.Tensor, stream=None) -> torch.Tensor:
        L.eat_ppl_trend(h, self.S, self.d, self.w, self.V, target, self.nll_sum, self.count, self.ppl_prev,
                        self.trend, self.nll, self.ws, self.ws.numel(), stream)
        return self.trend


def layerwise_caps(n_layers: int, lower: int, k_lower: int, k_upper: int):
    """Per-layer caps K for layer-wise sparsity: the paper's layer analysis
    (Sec. 4) finds lower layers' experts less critical than higher layers',
    so the lower ``lower`` layers get ``k_lower`` and the rest ``k_upper``."""
    return [k_lower if l < lower else k_upper for l in range(n_layers)]


class EatStack:
    """Stacked layers (one EatLayer each, own accounts) with their d x d
    mixing matrices, run one decode step at a time by eat_stack_forward."""

    def __init__(self, params, max_tokens: int, weights, mixes, device: str = "cuda"):
        self.layers = [EatLayer(p, max_tokens, w, device) for p, w in zip(params, weights)]
        self.mixes = list(mixes)
        self.device = torch.device(device)
        self._ws: Optional[torch.Tensor] = None
        self._arr = None

    def _entries(self):
        out = []
        for lay, m in zip(self.layers, self.mixes):
            w = lay.w
            out.append(L.eat_stack_layer_t(lay.handle, L._ptr(w["w_router"]), L._ptr(w["w1"]), L._ptr(w["w3"]),
                                           L._ptr(w["w2"]), L._ptr(w.get("ws1")), L._ptr(w.get("ws3")),
                                           L._ptr(w.get("ws2")), L._ptr(m), lay.acc))
        return L.stack_layers(out)

    def reset_accounts(self, stream=None) -> None:
        for lay in self.layers:
            lay.reset_accounts(stream)

    def forward(self, x: torch.Tensor, trend: Optional[torch.Tensor] = None, h_out: Optional[torch.Tensor] = None,
                masks_out: Optional[torch.Tensor] = None, probs_out: Optional[torch.Tensor] = None,
                rms_eps: float = 1e-6, stream=None) -> torch.Tensor:
        T = x.shape[0]
        if h_out is None:
            h_out = torch.empty_like(x)
        if self._arr is None:
            self._arr = self._entries()
        n = len(self.layers)
        need = L.eat_stack_workspace_size(self._arr, n, T)
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        L.eat_stack_forward(self._arr, n, x, T, trend, rms_eps, h_out, masks_out, probs_out, self._ws,
                            self._ws.numel(), stream)
        return h_out

    def close(self) -> None:
        for lay in self.layers:
            lay.close()


def capture(fn, warmup: int = 2) -> "torch.cuda.CUDAGraph":
    """Capture ``fn()`` -- calls into the library, which only enqueue on the
    current stream and never allocate or synchronise -- into a HIP graph.
    ``warmup`` eager calls first size every workspace (they run the layers,
    so reset accounts afterwards where that matters).  Replay with
    ``graph.replay()`` after copying new inputs into the tensors ``fn``
    reads; account updates inside the graph act on the live account
    tensors, so replays carry the history forward."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(warmup):
            fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    return g


def to_device(weights: Dict, device: str = "cuda") -> Dict[str, torch.Tensor]:
    """Upload generator output (fp32 arrays or bf16 bit patterns as uint16)
    to device tensors (torch.bfloat16 for bf16)."""
    import numpy as np
    out = {}
    for k, v in weights.items():
        t = torch.from_numpy(np.ascontiguousarray(v))
        if v.dtype == np.uint16:
            t = t.view(torch.bfloat16)
        out[k] = t.to(device)
    return out


# expert matrices and the (groups, M, K) view eat_pack_weights takes of each
_PACK_SHAPES = {"w1": ("E", "F", "d"), "w3": ("E", "F", "d"), "w2": ("E", "d", "F"),
                "ws1": (1, "Fs", "d"), "ws3": (1, "Fs", "d"), "ws2": (1, "d", "Fs")}


def pack_weights(weights: Dict[str, torch.Tensor], stream=None) -> Dict[str, torch.Tensor]:
    """Device weight dict -> the same dict with the bf16 expert matrices
    (w1, w3, w2 and the shared ws1, ws3, ws2) in the packed layout (new
    tensors, written by eat_pack_weights); for layers created with
    weight_layout = EAT_LAYOUT_PACKED.  Other entries are passed through."""
    out = dict(weights)
    for name, w in weights.items():
        if name not in _PACK_SHAPES or w is None:
            continue
        if w.dtype != torch.bfloat16 or w.dim() not in (2, 3):
            raise ValueError(f"{name}: packing needs a bf16 [groups][M][K] or [M][K] tensor")
        g, M, K = (1, *w.shape) if w.dim() == 2 else tuple(w.shape)
        dst = torch.empty_like(w)
        L.eat_pack_weights(w.contiguous(), g, M, K, dst, stream)
        out[name] = dst
    return out
