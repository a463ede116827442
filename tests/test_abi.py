"""C-ABI checks that need no GPU.

* libeat.so loads and exports every function include/eat.h declares;
* the ctypes mirror of eat_params_t / eat_accounts_t has the C layout
  (checked against a probe compiled with gcc from the header itself);
* eat_params_default fills the paper's hyper-parameter table;
* every validation path returns its status on the host, before any HIP
  call (these calls use fake addresses that are never dereferenced).
"""
import ctypes as C
import os
import re
import shutil
import subprocess

import pytest

import paper_2609_33614_amd as eat
from paper_2609_33614_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "eat.h")

pytestmark = pytest.mark.skipif(not os.path.exists(L.LIB_PATH), reason="libeat.so not built")


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(eat_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol():
    lib = C.CDLL(L.LIB_PATH)
    names = _declared_functions()
    assert {"eat_create", "eat_route", "eat_moe_forward", "eat_reset_accounts"} <= set(names)
    for n in names:
        assert hasattr(lib, n), f"{n} not exported"


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc missing")
def test_struct_layout_matches_header(tmp_path):
    fields = [f for f, _ in L.eat_params_t._fields_]
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "eat.h"', "int main(void){",
             'printf("%zu\\n", sizeof(eat_params_t));',
             'printf("%zu\\n", sizeof(eat_accounts_t));']
    for f in fields:
        lines.append(f'printf("%zu\\n", offsetof(eat_params_t, {f}));')
    sfields = [f for f, _ in L.eat_stack_layer_t._fields_]
    lines.append('printf("%zu\\n", sizeof(eat_stack_layer_t));')
    for f in sfields:
        lines.append(f'printf("%zu\\n", offsetof(eat_stack_layer_t, {f}));')
    lines.append("return 0;}")
    c = tmp_path / "probe.c"
    c.write_text("\n".join(lines))
    exe = tmp_path / "probe"
    r = subprocess.run(["gcc", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                        "-I", "/opt/rocm/include", str(c), "-o", str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    out = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True).stdout.split()]
    assert out[0] == C.sizeof(L.eat_params_t)
    assert out[1] == C.sizeof(L.eat_accounts_t)
    for f, off in zip(fields, out[2:]):
        assert getattr(L.eat_params_t, f).offset == off, f
    rest = out[2 + len(fields):]
    assert rest[0] == C.sizeof(L.eat_stack_layer_t)
    for f, off in zip(sfields, rest[1:]):
        assert getattr(L.eat_stack_layer_t, f).offset == off, f


def test_defaults_are_the_papers_table():
    p = eat.eat_params_default()
    assert p.mode == eat.EAT_MODE_EAT and p.top_k == 2
    expect = dict(alpha=0.95, w1=0.3, w2=0.3, w3=0.4, beta=0.6, alpha1=0.5, alpha2=1.0,
                  kappa1=0.7, kappa2=0.3, ppl_up=1.2, ppl_down=0.9, q_lo=0.1, q_hi=0.9, eps=1e-8,
                  inv_temperature=1.0)
    for k, v in expect.items():
        assert getattr(p, k) == pytest.approx(v, rel=1e-6), k
    assert p.cs_mode == 0 and p.d_shared == 0 and not p.expert_scale


def _params(**kw):
    base = dict(E=8, d_model=128, d_ffn=256, top_k=2, act_dtype=eat.EAT_F32, expert_dtype=eat.EAT_F32)
    base.update(kw)
    return eat.eat_params_default(**base)


@pytest.mark.parametrize("field,value,status", [
    ("E", 0, L.EAT_ERR_INVALID_ARG),
    ("E", 257, L.EAT_ERR_UNSUPPORTED),
    ("top_k", 0, L.EAT_ERR_INVALID_ARG),
    ("top_k", 9, L.EAT_ERR_INVALID_ARG),
    ("d_model", 100, L.EAT_ERR_UNSUPPORTED),
    ("d_ffn", 0, L.EAT_ERR_INVALID_ARG),
    ("d_shared", 96, L.EAT_ERR_UNSUPPORTED),
    ("alpha", 1.5, L.EAT_ERR_INVALID_ARG),
    ("beta", -0.1, L.EAT_ERR_INVALID_ARG),
    ("q_lo", 0.95, L.EAT_ERR_INVALID_ARG),
    ("inv_temperature", 0.0, L.EAT_ERR_INVALID_ARG),
    ("w3", float("nan"), L.EAT_ERR_INVALID_ARG),
    ("cs_mode", 2, L.EAT_ERR_INVALID_ARG),
    ("mode", 3, L.EAT_ERR_INVALID_ARG),
    ("act_dtype", 7, L.EAT_ERR_INVALID_ARG),
    ("expert_dtype", 1, L.EAT_ERR_UNSUPPORTED),
    ("top_p_cap", 9, L.EAT_ERR_INVALID_ARG),
    ("expert_scale", (1 << 20) + 2, L.EAT_ERR_INVALID_ARG),     # misaligned scale vector
    ("weight_layout", 2, L.EAT_ERR_INVALID_ARG),
    ("weight_layout", L.EAT_LAYOUT_PACKED, L.EAT_ERR_UNSUPPORTED),  # packed needs bf16 experts
    ("d_ffn", 32768 * 2, L.EAT_ERR_UNSUPPORTED),                   # d * F >= 2^31 with d = 32768 below
])
def test_create_rejects_bad_params(field, value, status):
    p = _params(**({field: value, "d_model": 32768} if field == "d_ffn" and value > 4096 else {field: value}))
    with pytest.raises(eat.EatError) as ei:
        eat.eat_create(p, 32)
    assert ei.value.status == status


@pytest.mark.parametrize("E", [64, 65, 128, 200, 256])
def test_create_accepts_up_to_256_experts(E):
    # masks are ceil(E / 64) words per token; 257 experts are rejected above
    h = eat.eat_create(_params(E=E, top_k=8), 128)
    try:
        assert L.mask_words(E) == (1 if E <= 64 else 2 if E <= 128 else 4)
        assert eat.eat_workspace_size(h, 128) > eat.eat_workspace_size(h, 1) > 0
    finally:
        eat.eat_destroy(h)


def test_create_rejects_bad_top_p_and_token_limits():
    with pytest.raises(eat.EatError):
        eat.eat_create(_params(mode=eat.EAT_MODE_TOPP, top_p=0.0), 32)
    with pytest.raises(eat.EatError):
        eat.eat_create(_params(mode=eat.EAT_MODE_TOPP, top_p=1.5), 32)
    for bad in (0, -1, (1 << 24) + 1):
        with pytest.raises(eat.EatError):
            eat.eat_create(_params(), bad)


def test_create_rejects_row_counts_past_32_bits():
    # selected rows are indexed with int32: max_tokens * (most experts per token) < 2^31
    with pytest.raises(eat.EatError) as ei:
        eat.eat_create(_params(E=256, top_k=8), 1 << 23)          # EAT keeps up to E per token
    assert ei.value.status == L.EAT_ERR_UNSUPPORTED
    with pytest.raises(eat.EatError) as ei:
        eat.eat_create(_params(mode=eat.EAT_MODE_TOPP, E=256, top_k=8), 1 << 23)
    assert ei.value.status == L.EAT_ERR_UNSUPPORTED
    for p in (_params(mode=eat.EAT_MODE_TOPK, E=256, top_k=8),     # K rows per token
              _params(mode=eat.EAT_MODE_TOPP, E=256, top_k=8, top_p_cap=8),
              _params(E=64, top_k=8)):
        h = eat.eat_create(p, 1 << 23 if p.E == 256 else (1 << 24) - 1)
        eat.eat_destroy(h)


def test_workspace_grows_with_tokens_and_mode():
    h_eat = eat.eat_create(_params(), 1024)
    h_topk = eat.eat_create(_params(mode=eat.EAT_MODE_TOPK), 1024)
    try:
        sizes = [eat.eat_workspace_size(h_eat, T) for T in (0, 1, 16, 1024)]
        assert sizes == sorted(sizes) and sizes[-1] > sizes[0]
        # EAT keeps exact ties (up to E per token), Top-K exactly K
        assert eat.eat_workspace_size(h_eat, 1024) > eat.eat_workspace_size(h_topk, 1024)
        with pytest.raises(eat.EatError):
            eat.eat_workspace_size(h_eat, 1025)
        with pytest.raises(eat.EatError):
            eat.eat_workspace_size(h_eat, -1)
    finally:
        eat.eat_destroy(h_eat)
        eat.eat_destroy(h_topk)


FAKE = 1 << 20          # 16-byte (and 256-byte) aligned fake address, never dereferenced


def _fwd(h, **kw):
    args = dict(x=FAKE, T=4, w_router=FAKE, w1=FAKE, w3=FAKE, w2=FAKE, ws1=None, ws3=None, ws2=None,
                acc=L.accounts(FAKE, FAKE, FAKE), ppl_trend=None, y=FAKE, mask_out=None,
                expert_load_out=None, ws=FAKE, ws_bytes=0, stream=0)
    args.update(kw)
    eat.eat_moe_forward(h, **args)


def test_forward_validation_happens_on_the_host():
    h = eat.eat_create(_params(), 64)
    try:
        need = eat.eat_workspace_size(h, 4)
        cases = [
            (dict(x=None, ws_bytes=need), L.EAT_ERR_INVALID_ARG),
            (dict(w2=None, ws_bytes=need), L.EAT_ERR_INVALID_ARG),
            (dict(y=None, ws_bytes=need), L.EAT_ERR_INVALID_ARG),
            (dict(x=FAKE + 4, ws_bytes=need), L.EAT_ERR_INVALID_ARG),          # misaligned
            (dict(T=65, ws_bytes=need), L.EAT_ERR_INVALID_ARG),                # > max_tokens
            (dict(T=-1, ws_bytes=need), L.EAT_ERR_INVALID_ARG),
            (dict(acc=L.accounts(None, FAKE, FAKE), ws_bytes=need), L.EAT_ERR_INVALID_ARG),
            (dict(ws1=FAKE, ws_bytes=need), L.EAT_ERR_INVALID_ARG),            # no shared expert declared
            (dict(ws_bytes=need - 1), L.EAT_ERR_WORKSPACE),
            (dict(ws=None, ws_bytes=need), L.EAT_ERR_WORKSPACE),
            (dict(ws=FAKE + 16, ws_bytes=need), L.EAT_ERR_INVALID_ARG),        # workspace not 256-aligned
            (dict(mask_out=FAKE + 4, ws_bytes=need), L.EAT_ERR_INVALID_ARG),
        ]
        for kw, status in cases:
            with pytest.raises(eat.EatError) as ei:
                _fwd(h, **kw)
            assert ei.value.status == status, kw
        # an empty call is valid and launches nothing
        _fwd(h, T=0, ws=None, ws_bytes=0)
    finally:
        eat.eat_destroy(h)


def test_noalloc_forward_validation_happens_on_the_host():
    """The allocation-free forward checks its arguments like eat_moe_forward
    and rejects a call that needs more than its fixed scratch array, all on
    the host before any HIP call."""
    def noalloc(h, **kw):
        args = dict(x=FAKE, T=4, w_router=FAKE, w1=FAKE, w3=FAKE, w2=FAKE, ws1=None, ws3=None, ws2=None,
                    acc=L.accounts(FAKE, FAKE, FAKE), ppl_trend=None, y=FAKE, mask_out=None, expert_load_out=None,
                    stream=0)
        args.update(kw)
        eat.eat_moe_forward_noalloc(h, **args)

    # the fine-grained EAT layer at 256 tokens needs ~545 MB: above the limit
    p = _params(E=64, d_model=2048, d_ffn=1024, top_k=8, act_dtype=eat.EAT_BF16, expert_dtype=eat.EAT_BF16)
    h = eat.eat_create(p, 256)
    try:
        assert eat.eat_workspace_size(h, 256) > eat.EAT_NOALLOC_SCRATCH_BYTES
        assert eat.eat_workspace_size(h, 16) <= eat.EAT_NOALLOC_SCRATCH_BYTES
        for kw, status in [(dict(T=256), L.EAT_ERR_SCRATCH_LIMIT), (dict(x=None), L.EAT_ERR_INVALID_ARG),
                           (dict(y=FAKE + 4), L.EAT_ERR_INVALID_ARG), (dict(T=257), L.EAT_ERR_INVALID_ARG),
                           (dict(acc=L.accounts(FAKE, None, FAKE)), L.EAT_ERR_INVALID_ARG)]:
            with pytest.raises(eat.EatError) as ei:
                noalloc(h, **kw)
            assert ei.value.status == status, kw
        noalloc(h, T=0)                  # an empty call is valid and launches nothing
    finally:
        eat.eat_destroy(h)


def test_shared_expert_pointers_required_when_declared():
    h = eat.eat_create(_params(d_shared=128), 8)
    try:
        with pytest.raises(eat.EatError) as ei:
            _fwd(h, ws_bytes=eat.eat_workspace_size(h, 4))
        assert ei.value.status == L.EAT_ERR_INVALID_ARG
    finally:
        eat.eat_destroy(h)


def test_baseline_modes_need_no_accounts():
    h = eat.eat_create(_params(mode=eat.EAT_MODE_TOPK), 8)
    try:
        # null accounts pass validation in Top-K; the empty call launches nothing
        _fwd(h, T=0, acc=L.accounts(None, None, None), ws=None)
    finally:
        eat.eat_destroy(h)


def test_route_validation_happens_on_the_host():
    h = eat.eat_create(_params(), 16)
    try:
        need = eat.eat_route_workspace_size(h, 4)
        assert 0 < need <= eat.eat_workspace_size(h, 4)
        base = dict(x=FAKE, T=4, w_router=FAKE, acc=L.accounts(FAKE, FAKE, FAKE), ppl_trend=None,
                    mask_out=FAKE, k_out=FAKE, gate_out=FAKE, prob_out=None, ws=FAKE, ws_bytes=need, stream=0)
        for kw, status in ((dict(ws=None), L.EAT_ERR_WORKSPACE), (dict(ws_bytes=need - 1), L.EAT_ERR_WORKSPACE),
                           (dict(ws=FAKE + 64), L.EAT_ERR_INVALID_ARG)):
            args = dict(base); args.update(kw)
            with pytest.raises(eat.EatError) as ei:
                eat.eat_route(h, **args)
            assert ei.value.status == status, kw
        for kw in (dict(mask_out=None), dict(k_out=None), dict(gate_out=None), dict(x=None),
                   dict(w_router=FAKE + 8), dict(T=17), dict(acc=L.accounts(FAKE, None, FAKE))):
            args = dict(base); args.update(kw)
            with pytest.raises(eat.EatError) as ei:
                eat.eat_route(h, **args)
            assert ei.value.status == L.EAT_ERR_INVALID_ARG, kw
        args = dict(base); args.update(T=0, ws=None, ws_bytes=0)
        eat.eat_route(h, **args)
        with pytest.raises(eat.EatError):
            eat.eat_reset_accounts(h, L.accounts(None, FAKE, FAKE), 0)
    finally:
        eat.eat_destroy(h)


def test_status_strings():
    for s in range(6):
        assert isinstance(eat.eat_status_string(s), str) and eat.eat_status_string(s)
    assert eat.eat_status_string(99) == "unknown status"


def _stack_entry(h, **kw):
    e = dict(layer=h, w_router=FAKE, w1=FAKE, w3=FAKE, w2=FAKE, ws1=None, ws3=None, ws2=None, mix=FAKE,
             acc=L.accounts(FAKE, FAKE, FAKE))
    e.update(kw)
    return L.eat_stack_layer_t(e["layer"], e["w_router"], e["w1"], e["w3"], e["w2"], e["ws1"], e["ws3"], e["ws2"],
                               e["mix"], e["acc"])


def test_stack_validation_happens_on_the_host():
    bf = dict(act_dtype=eat.EAT_BF16, expert_dtype=eat.EAT_BF16)
    hs = [eat.eat_create(_params(**bf), 16) for _ in range(3)]
    h_f32 = eat.eat_create(_params(), 16)
    h_d256 = eat.eat_create(_params(d_model=256, **bf), 16)
    try:
        arr = L.stack_layers([_stack_entry(h) for h in hs])
        need = eat.eat_stack_workspace_size(arr, 3, 4)
        assert need > eat.eat_workspace_size(hs[0], 4)
        assert eat.eat_stack_workspace_size(arr, 3, 8) > need
        base = dict(x=FAKE, T=4, ppl_trend=None, rms_eps=1e-6, h_out=FAKE, masks_out=None, probs_out=None, ws=FAKE,
                    ws_bytes=need, stream=0)
        cases = [
            (dict(n_layers=0), L.EAT_ERR_INVALID_ARG),
            (dict(T=17), L.EAT_ERR_INVALID_ARG),                      # above the layers' max_tokens
            (dict(x=None), L.EAT_ERR_INVALID_ARG),
            (dict(h_out=FAKE + 8), L.EAT_ERR_INVALID_ARG),
            (dict(rms_eps=-1.0), L.EAT_ERR_INVALID_ARG),
            (dict(rms_eps=float("nan")), L.EAT_ERR_INVALID_ARG),
            (dict(ws_bytes=need - 1), L.EAT_ERR_WORKSPACE),
            (dict(ws=FAKE + 128), L.EAT_ERR_INVALID_ARG),
            (dict(masks_out=FAKE + 4), L.EAT_ERR_INVALID_ARG),
            (dict(probs_out=FAKE + 2), L.EAT_ERR_INVALID_ARG),
        ]
        for kw, status in cases:
            args = dict(base, n_layers=3); args.update(kw)
            with pytest.raises(eat.EatError) as ei:
                eat.eat_stack_forward(arr, **args)
            assert ei.value.status == status, kw
        bad_layers = [
            ([_stack_entry(hs[0]), _stack_entry(h_f32)], L.EAT_ERR_UNSUPPORTED),      # fp32 layer
            ([_stack_entry(hs[0]), _stack_entry(h_d256)], L.EAT_ERR_INVALID_ARG),     # different d_model
            ([_stack_entry(hs[0], mix=None)], L.EAT_ERR_INVALID_ARG),
            ([_stack_entry(hs[0], mix=FAKE + 2)], L.EAT_ERR_INVALID_ARG),
            ([_stack_entry(hs[0], w2=None)], L.EAT_ERR_INVALID_ARG),
            ([_stack_entry(hs[0], acc=L.accounts(FAKE, None, FAKE))], L.EAT_ERR_INVALID_ARG),
            ([_stack_entry(hs[0], ws1=FAKE)], L.EAT_ERR_INVALID_ARG),                 # no shared expert declared
            ([_stack_entry(None)], L.EAT_ERR_INVALID_ARG),
        ]
        for entries, status in bad_layers:
            a2 = L.stack_layers(entries)
            with pytest.raises(eat.EatError) as ei:
                eat.eat_stack_forward(a2, len(entries), FAKE, 4, None, 1e-6, FAKE, None, None, FAKE, 1 << 40, stream=0)
            assert ei.value.status == status
        # an empty step is valid and launches nothing
        eat.eat_stack_forward(arr, 3, FAKE, 0, None, 1e-6, FAKE, None, None, None, 0, stream=0)
    finally:
        for h in hs + [h_f32, h_d256]:
            eat.eat_destroy(h)


def test_ppl_validation_happens_on_the_host():
    need = eat.eat_ppl_workspace_size(4, 128, 256)
    assert need >= 4 * 256 * 4
    for args in ((-1, 128, 256), (4, 100, 256), (4, 128, 100), (4, 0, 256), (4, 128, 0)):
        with pytest.raises(eat.EatError):
            eat.eat_ppl_workspace_size(*args)
    base = dict(h=FAKE, S=4, d=128, w_vocab=FAKE, V=256, target=FAKE, nll_sum=FAKE, count=FAKE, ppl_prev=FAKE,
                trend_out=FAKE, nll_out=None, ws=FAKE, ws_bytes=need, stream=0)
    cases = [(dict(h=None), L.EAT_ERR_INVALID_ARG), (dict(target=None), L.EAT_ERR_INVALID_ARG),
             (dict(h=FAKE + 8), L.EAT_ERR_INVALID_ARG), (dict(nll_sum=FAKE + 4), L.EAT_ERR_INVALID_ARG),
             (dict(V=100), L.EAT_ERR_INVALID_ARG), (dict(ws_bytes=need - 1), L.EAT_ERR_WORKSPACE),
             (dict(ws=None), L.EAT_ERR_WORKSPACE), (dict(ws=FAKE + 64), L.EAT_ERR_INVALID_ARG)]
    for kw, status in cases:
        args = dict(base); args.update(kw)
        with pytest.raises(eat.EatError) as ei:
            eat.eat_ppl_trend(**args)
        assert ei.value.status == status, kw
    args = dict(base); args.update(S=0, h=None, ws=None, ws_bytes=0)
    eat.eat_ppl_trend(**args)
    with pytest.raises(eat.EatError):
        eat.eat_ppl_reset(4, None, FAKE, FAKE, stream=0)


def test_packed_layout_accepted_for_bf16_experts():
    h = eat.eat_create(_params(act_dtype=eat.EAT_BF16, expert_dtype=eat.EAT_BF16, weight_layout=L.EAT_LAYOUT_PACKED),
                       16)
    eat.eat_destroy(h)


def test_pack_validation_happens_on_the_host():
    ok = dict(src=FAKE, groups=2, M=64, K=128, dst=FAKE + (1 << 24), stream=0)
    cases = [dict(src=None), dict(dst=None), dict(groups=0), dict(M=40), dict(K=48), dict(M=0),
             dict(src=FAKE + 8), dict(dst=FAKE + (1 << 24) + 2),
             dict(dst=FAKE + 1024)]                                   # overlaps src
    for kw in cases:
        args = dict(ok); args.update(kw)
        with pytest.raises(eat.EatError) as ei:
            eat.eat_pack_weights(**args)
        assert ei.value.status == L.EAT_ERR_INVALID_ARG, kw


def test_binding_rejects_host_and_strided_tensors():
    # the C entry points take dense device arrays; the binding refuses what
    # they could not check (a host tensor would be read as a device address)
    import torch
    with pytest.raises(ValueError, match="device arrays"):
        L._ptr(torch.zeros(4))
    assert L._ptr(None) is None and L._ptr(FAKE) == FAKE
