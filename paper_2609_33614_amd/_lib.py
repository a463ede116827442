"""ctypes binding of libeat.so (include/eat.h).

Argument marshalling only: every function here has the name of the C entry
point it wraps, turns torch tensors into device pointers and the current
torch stream into a hipStream_t, and raises ``EatError`` on a non-OK status.
All computation happens in the library's HIP kernels; there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("EAT_LIB_PATH") or os.path.join(_HERE, "libeat.so")

(EAT_OK, EAT_ERR_INVALID_ARG, EAT_ERR_UNSUPPORTED, EAT_ERR_WORKSPACE, EAT_ERR_HIP, EAT_ERR_INTERNAL,
 EAT_ERR_SCRATCH_LIMIT) = range(7)
EAT_NOALLOC_SCRATCH_BYTES = 256 << 20      # include/eat.h
EAT_MODE_EAT, EAT_MODE_TOPK, EAT_MODE_TOPP = 0, 1, 2
EAT_F32, EAT_BF16 = 0, 1
EAT_LAYOUT_ROWS, EAT_LAYOUT_PACKED = 0, 1
(EAT_STAGE_BEGIN, EAT_STAGE_ROUTED, EAT_STAGE_PERMUTED, EAT_STAGE_UP, EAT_STAGE_DOWN, EAT_STAGE_SHARED,
 EAT_STAGE_COMBINED, EAT_STAGE_END, EAT_NUM_STAGE_EVENTS) = range(9)
MODES = {"eat": EAT_MODE_EAT, "topk": EAT_MODE_TOPK, "topp": EAT_MODE_TOPP}


class EatError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {eat_status_string(status)} (status {status})")


class eat_params_t(C.Structure):
    _fields_ = [
        ("mode", C.c_int32), ("E", C.c_int32), ("d_model", C.c_int32), ("d_ffn", C.c_int32),
        ("top_k", C.c_int32), ("top_p", C.c_float), ("top_p_cap", C.c_int32),
        ("alpha", C.c_float), ("w1", C.c_float), ("w2", C.c_float), ("w3", C.c_float),
        ("beta", C.c_float), ("alpha1", C.c_float), ("alpha2", C.c_float),
        ("kappa1", C.c_float), ("kappa2", C.c_float), ("ppl_up", C.c_float), ("ppl_down", C.c_float),
        ("q_lo", C.c_float), ("q_hi", C.c_float), ("eps", C.c_float), ("inv_temperature", C.c_float),
        ("cs_mode", C.c_int32), ("act_dtype", C.c_int32), ("expert_dtype", C.c_int32),
        ("d_shared", C.c_int32), ("expert_scale", C.c_void_p), ("weight_layout", C.c_int32),
    ]


class eat_accounts_t(C.Structure):
    _fields_ = [("n", C.c_void_p), ("p_total", C.c_void_p), ("c_s", C.c_void_p)]


class eat_stack_layer_t(C.Structure):
    _fields_ = [("layer", C.c_void_p), ("w_router", C.c_void_p), ("w1", C.c_void_p), ("w3", C.c_void_p),
                ("w2", C.c_void_p), ("ws1", C.c_void_p), ("ws3", C.c_void_p), ("ws2", C.c_void_p),
                ("mix", C.c_void_p), ("acc", eat_accounts_t)]


_lib = None


def load() -> C.CDLL:
    """Load libeat.so from the package directory.  Raises if it was not
    built (run ``python -m paper_2609_33614_amd.build``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_33614_amd.build`")
    lib = C.CDLL(LIB_PATH)
    st = C.c_int
    P = C.c_void_p
    lib.eat_params_default.argtypes = [C.POINTER(eat_params_t)]
    lib.eat_create.argtypes = [C.POINTER(eat_params_t), C.c_int32, C.POINTER(C.c_void_p)]
    lib.eat_destroy.argtypes = [P]
    lib.eat_workspace_size.argtypes = [P, C.c_int32, C.POINTER(C.c_size_t)]
    lib.eat_reset_accounts.argtypes = [P, eat_accounts_t, P]
    if hasattr(lib, "eat_route_workspace_size"):
        lib.eat_route_workspace_size.argtypes = [P, C.c_int32, C.POINTER(C.c_size_t)]
    lib.eat_route.argtypes = [P, P, C.c_int32, P, eat_accounts_t, P, P, P, P, P, P, C.c_size_t, P]
    lib.eat_moe_forward.argtypes = [P, P, C.c_int32, P, P, P, P, P, P, P, eat_accounts_t, P, P, P, P, P,
                                    C.c_size_t, P]
    lib.eat_moe_forward_profiled.argtypes = lib.eat_moe_forward.argtypes + [P, C.c_int32]
    if hasattr(lib, "eat_stack_forward"):
        lib.eat_stack_workspace_size.argtypes = [P, C.c_int32, C.c_int32, C.POINTER(C.c_size_t)]
        lib.eat_stack_forward.argtypes = [P, C.c_int32, P, C.c_int32, P, C.c_float, P, P, P, P, C.c_size_t, P]
    if hasattr(lib, "eat_ppl_trend"):
        lib.eat_ppl_workspace_size.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.POINTER(C.c_size_t)]
        lib.eat_ppl_reset.argtypes = [C.c_int32, P, P, P, P]
        lib.eat_ppl_trend.argtypes = [P, C.c_int32, C.c_int32, P, C.c_int32, P, P, P, P, P, P, P, C.c_size_t, P]
    if hasattr(lib, "eat_pack_weights"):
        lib.eat_pack_weights.argtypes = [P, C.c_int32, C.c_int32, C.c_int32, P, P]
    if hasattr(lib, "eat_moe_forward_noalloc"):
        lib.eat_moe_forward_noalloc.argtypes = lib.eat_moe_forward.argtypes[:15] + [P]
    lib.eat_status_string.argtypes = [C.c_int]
    lib.eat_status_string.restype = C.c_char_p
    for name in ("eat_params_default", "eat_create", "eat_destroy", "eat_workspace_size", "eat_route_workspace_size",
                 "eat_reset_accounts", "eat_route", "eat_moe_forward", "eat_moe_forward_profiled",
                 "eat_stack_workspace_size", "eat_stack_forward", "eat_ppl_workspace_size", "eat_ppl_reset",
                 "eat_ppl_trend", "eat_pack_weights", "eat_moe_forward_noalloc"):
        if hasattr(lib, name):
            getattr(lib, name).restype = st
    _lib = lib
    return lib


# ------------------------------------------------------------ marshalling --

def _ptr(t) -> Optional[int]:
    """Device address of a tensor (which must be a dense GPU tensor: the C
    entry points take device pointers to densely packed arrays and cannot
    check either), an int address, or None."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError("libeat takes device arrays: got a tensor on " + str(t.device))
    if not t.is_contiguous():
        raise ValueError("libeat takes densely packed arrays: got a non-contiguous tensor view")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(status: int, where: str):
    if status != EAT_OK:
        raise EatError(status, where)


def accounts(n=None, p_total=None, c_s=None) -> eat_accounts_t:
    return eat_accounts_t(_ptr(n), _ptr(p_total), _ptr(c_s))


def mask_words(E: int) -> int:
    """64-bit words of one token's selection mask (the ABI's [T][W] layout)."""
    return (int(E) + 63) // 64


# -------------------------------------------------------------- entry points --

def eat_status_string(status: int) -> str:
    return load().eat_status_string(int(status)).decode()


def eat_params_default(**overrides) -> eat_params_t:
    p = eat_params_t()
    _check(load().eat_params_default(C.byref(p)), "eat_params_default")
    for k, v in overrides.items():
        if k == "mode" and isinstance(v, str):
            v = MODES[v]
        setattr(p, k, v)
    return p


def eat_create(params: eat_params_t, max_tokens: int) -> int:
    h = C.c_void_p()
    _check(load().eat_create(C.byref(params), int(max_tokens), C.byref(h)), "eat_create")
    return h.value


def eat_destroy(handle: int) -> None:
    _check(load().eat_destroy(handle), "eat_destroy")


def eat_workspace_size(handle: int, T: int) -> int:
    b = C.c_size_t()
    _check(load().eat_workspace_size(handle, int(T), C.byref(b)), "eat_workspace_size")
    return b.value


def eat_route_workspace_size(handle: int, T: int) -> int:
    b = C.c_size_t()
    _check(load().eat_route_workspace_size(handle, int(T), C.byref(b)), "eat_route_workspace_size")
    return b.value


def eat_reset_accounts(handle: int, acc: eat_accounts_t, stream=None) -> None:
    _check(load().eat_reset_accounts(handle, acc, _stream(stream)), "eat_reset_accounts")


def eat_route(handle: int, x, T: int, w_router, acc: eat_accounts_t, ppl_trend, mask_out, k_out,
              gate_out, prob_out=None, ws=None, ws_bytes: int = 0, stream=None) -> None:
    _check(load().eat_route(handle, _ptr(x), int(T), _ptr(w_router), acc, _ptr(ppl_trend), _ptr(mask_out),
                            _ptr(k_out), _ptr(gate_out), _ptr(prob_out), _ptr(ws), int(ws_bytes),
                            _stream(stream)), "eat_route")


def eat_moe_forward(handle: int, x, T: int, w_router, w1, w3, w2, ws1, ws3, ws2, acc: eat_accounts_t,
                    ppl_trend, y, mask_out, expert_load_out, ws, ws_bytes: int, stream=None) -> None:
    _check(load().eat_moe_forward(handle, _ptr(x), int(T), _ptr(w_router), _ptr(w1), _ptr(w3), _ptr(w2),
                                  _ptr(ws1), _ptr(ws3), _ptr(ws2), acc, _ptr(ppl_trend), _ptr(y),
                                  _ptr(mask_out), _ptr(expert_load_out), _ptr(ws), int(ws_bytes),
                                  _stream(stream)), "eat_moe_forward")


def eat_moe_forward_profiled(handle: int, x, T: int, w_router, w1, w3, w2, ws1, ws3, ws2,
                             acc: eat_accounts_t, ppl_trend, y, mask_out, expert_load_out, ws,
                             ws_bytes: int, stream=None, events=None) -> None:
    """``events``: sequence of hipEvent_t handles (ints) or None, indexed by
    stage boundary (EAT_STAGE_*)."""
    events = list(events or [])
    arr = (C.c_void_p * max(1, len(events)))(*[e or None for e in events]) if events else None
    _check(load().eat_moe_forward_profiled(handle, _ptr(x), int(T), _ptr(w_router), _ptr(w1), _ptr(w3),
                                           _ptr(w2), _ptr(ws1), _ptr(ws3), _ptr(ws2), acc, _ptr(ppl_trend),
                                           _ptr(y), _ptr(mask_out), _ptr(expert_load_out), _ptr(ws),
                                           int(ws_bytes), _stream(stream), arr, len(events)),
           "eat_moe_forward_profiled")


def eat_moe_forward_noalloc(handle: int, x, T: int, w_router, w1, w3, w2, ws1, ws3, ws2, acc: eat_accounts_t,
                            ppl_trend, y, mask_out, expert_load_out, stream=None) -> None:
    _check(load().eat_moe_forward_noalloc(handle, _ptr(x), int(T), _ptr(w_router), _ptr(w1), _ptr(w3), _ptr(w2),
                                          _ptr(ws1), _ptr(ws3), _ptr(ws2), acc, _ptr(ppl_trend), _ptr(y),
                                          _ptr(mask_out), _ptr(expert_load_out), _stream(stream)),
           "eat_moe_forward_noalloc")


def stack_layers(entries) -> "C.Array":
    """Host array of eat_stack_layer_t from a sequence of eat_stack_layer_t."""
    entries = list(entries)
    return (eat_stack_layer_t * len(entries))(*entries)


def eat_stack_workspace_size(layers, n_layers: int, T: int) -> int:
    b = C.c_size_t()
    _check(load().eat_stack_workspace_size(C.cast(layers, C.c_void_p) if layers is not None else None,
                                           int(n_layers), int(T), C.byref(b)), "eat_stack_workspace_size")
    return b.value


def eat_stack_forward(layers, n_layers: int, x, T: int, ppl_trend, rms_eps: float, h_out, masks_out, probs_out,
                      ws, ws_bytes: int, stream=None) -> None:
    _check(load().eat_stack_forward(C.cast(layers, C.c_void_p) if layers is not None else None, int(n_layers),
                                    _ptr(x), int(T), _ptr(ppl_trend), float(rms_eps), _ptr(h_out),
                                    _ptr(masks_out), _ptr(probs_out), _ptr(ws), int(ws_bytes), _stream(stream)),
           "eat_stack_forward")


def eat_ppl_workspace_size(S: int, d: int, V: int) -> int:
    b = C.c_size_t()
    _check(load().eat_ppl_workspace_size(int(S), int(d), int(V), C.byref(b)), "eat_ppl_workspace_size")
    return b.value


def eat_ppl_reset(S: int, nll_sum, count, ppl_prev, stream=None) -> None:
    _check(load().eat_ppl_reset(int(S), _ptr(nll_sum), _ptr(count), _ptr(ppl_prev), _stream(stream)), "eat_ppl_reset")


def eat_ppl_trend(h, S: int, d: int, w_vocab, V: int, target, nll_sum, count, ppl_prev, trend_out, nll_out, ws,
                  ws_bytes: int, stream=None) -> None:
    _check(load().eat_ppl_trend(_ptr(h), int(S), int(d), _ptr(w_vocab), int(V), _ptr(target), _ptr(nll_sum),
                                _ptr(count), _ptr(ppl_prev), _ptr(trend_out), _ptr(nll_out), _ptr(ws), int(ws_bytes),
                                _stream(stream)), "eat_ppl_trend")


def eat_pack_weights(src, groups: int, M: int, K: int, dst, stream=None) -> None:
    _check(load().eat_pack_weights(_ptr(src), int(groups), int(M), int(K), _ptr(dst), _stream(stream)),
           "eat_pack_weights")
