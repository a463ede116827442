"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Same seeded inputs on both sides; every account state either starts at
zero or comes from the seeded generator, never from the GPU.  Checks:
router probabilities and gates within TOL_P; selection masks bit-exact for
every non-borderline token; layer outputs within the per-token relative
tolerance; account updates (N exact, P_total / C_s relative).
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_33614_amd import _lib as L
from paper_2609_33614_amd.layer import EatLayer, to_device
from tests import parity as PT
from workload import (SHAPES, HiddenStream, make_accounts, make_expert_scale, make_layer_weights, make_prefill,
                      make_trend)

pytestmark = pytest.mark.gpu

MODES = {"eat": O.MODE_EAT, "topk": O.MODE_TOPK, "topp": O.MODE_TOPP}

# reduced shapes: several tiles in every dimension and ragged token tails
SMALL = {
    "tiny": dict(shape="tiny", d=128, F=256, E=8, Fs=0),
    "mixtral": dict(shape="mixtral", d=512, F=768, E=8, Fs=0),
    "finegrained": dict(shape="finegrained", d=256, F=256, E=64, Fs=0),
    "shared": dict(shape="shared", d=256, F=192, E=60, Fs=320),
    # an always-on expert wide enough that both of its projections split
    # their reduction dimension (up/gate in 2 slices, down in 8)
    "shared_split": dict(shape="shared", d=256, F=192, E=60, Fs=1024),
    # more than 64 experts: masks of 2-4 words, ragged last words
    "tiny_e100": dict(shape="tiny", d=128, F=128, E=100, Fs=0),
    "qwen3": dict(shape="qwen3", d=256, F=256, E=128, Fs=0),
    "qwen3_e200": dict(shape="qwen3", d=128, F=128, E=200, Fs=0),
    "qwen3_e256": dict(shape="qwen3", d=128, F=192, E=256, Fs=0),
}
WIDE_E = ["tiny_e100", "qwen3", "qwen3_e200", "qwen3_e256"]


def _x_host(shape, T, d, seed):
    return HiddenStream(shape, T, seed=seed, d=d).next()


def _x_dev(x_host):
    t = torch.from_numpy(np.ascontiguousarray(x_host))
    if x_host.dtype == np.uint16:
        t = t.view(torch.bfloat16)
    return t.cuda()


def _y_host(y):
    return y.float().cpu().numpy().astype(np.float64)


def _layer(case, mode, K=None, top_p=None, cs_mode=0, max_tokens=512, seed=None, scale=None, top_p_cap=0):
    shape = SHAPES[case["shape"]]
    w = make_layer_weights(shape, seed=seed, E=case["E"], d=case["d"], F=case["F"], F_shared=case["Fs"])
    dt = L.EAT_BF16 if shape.bf16 else L.EAT_F32
    p = L.eat_params_default(mode=MODES[mode], E=case["E"], d_model=case["d"], d_ffn=case["F"],
                             top_k=shape.K if K is None else K,
                             top_p=(shape.top_p or 0.6) if top_p is None else top_p,
                             inv_temperature=shape.inv_temp, cs_mode=cs_mode, act_dtype=dt,
                             expert_dtype=dt, d_shared=case["Fs"], top_p_cap=top_p_cap)
    scale_dev = None
    if scale is not None:
        scale_dev = torch.from_numpy(scale).cuda()
        p.expert_scale = scale_dev.data_ptr()
    lay = EatLayer(p, max_tokens, to_device(w))
    lay.scale_dev = scale_dev            # the handle keeps the pointer: keep the tensor alive
    prm = PT.oracle_params(shape, MODES[mode], K=K, top_p=top_p, cs_mode=cs_mode, shared=case["Fs"] > 0)
    prm.expert_scale = scale
    prm.top_p_cap = top_p_cap
    return shape, w, lay, prm


def _check_routing(name, r, prm, mask, gate, prob, k):
    border = PT.borderline(r, prm)
    gm = PT.masks_to_list(mask)
    bad = [t for t in range(len(gm)) if not border[t] and gm[t] != r.masks[t]]
    dp = np.abs(prob.cpu().numpy() - r.p).max()
    ok_rows = ~border
    dg = np.abs(gate.cpu().numpy()[ok_rows] - r.g_norm[ok_rows]).max() if ok_rows.any() else 0.0
    kk = k.cpu().numpy()
    PT.report(name, T=len(gm), borderline=int(border.sum()), mask_mismatch=len(bad), max_dp=f"{dp:.2e}",
              max_dgate=f"{dg:.2e}", mean_k=f"{kk.mean():.3f}")
    assert not bad, f"{len(bad)} non-borderline mask mismatches, e.g. token {bad[0]}"
    assert dp <= PT.TOL_P
    assert dg <= PT.TOL_P
    assert (kk[ok_rows] == r.k[ok_rows]).all()
    if prm.mode == O.MODE_EAT:
        # the band must cover the observed importance error, |dI| ~ (1 - beta) |dp|
        assert 4 * (1 - prm.beta) * dp <= PT.EPS_B
    return border


# ------------------------------------------------------------------ routing --

@pytest.mark.parametrize("case", ["tiny", "mixtral", "finegrained", "shared"] + WIDE_E)
@pytest.mark.parametrize("mode", ["eat", "topk", "topp"])
@pytest.mark.parametrize("T", [1, 37, 300])
def test_route_parity(case, mode, T):
    c = SMALL[case]
    shape, w, lay, prm = _layer(c, mode)
    x = _x_host(shape, T, c["d"], seed=T)
    trend = make_trend(T, seed=T)
    acc = make_accounts(c["E"], seed=T + 1)
    if mode == "eat":
        lay.load_accounts(*acc)
    mask, k, gate, prob = lay.route(_x_dev(x), torch.from_numpy(trend).cuda())
    torch.cuda.synchronize()
    r = O.route(x, w["w_router"], acc, trend, prm)
    _check_routing(f"route {case} {mode} T={T}", r, prm, mask, gate, prob, k)


@pytest.mark.parametrize("case", ["tiny", "mixtral", "finegrained"])
@pytest.mark.parametrize("mode", ["eat", "topk", "topp"])
def test_opd_reweighting_parity(case, mode):
    """Sec. 3.5: per-expert scales applied to p before selection (routing,
    gates, probabilities, and the forward's accounts)."""
    c = SMALL[case]
    T = 200
    scale = make_expert_scale(c["E"], seed=17)
    shape, w, lay, prm = _layer(c, mode, scale=scale)
    x = _x_host(shape, T, c["d"], seed=55)
    acc = make_accounts(c["E"], seed=3, c_scale=0.05)
    if mode == "eat":
        lay.load_accounts(*acc)
    mask, k, gate, prob = lay.route(_x_dev(x))
    torch.cuda.synchronize()
    r = O.route(x, w["w_router"], acc, None, prm)
    _check_routing(f"opd route {case} {mode} T={T}", r, prm, mask, gate, prob, k)
    # the scales change the selection of some tokens (the hook is live)
    plain = O.route(x, w["w_router"], acc, None, PT.oracle_params(shape, MODES[mode]))
    assert sum(a != b for a, b in zip(plain.masks, r.masks)) > 0
    # forward: y and the account update use the reweighted probabilities
    y = lay.forward(_x_dev(x), mask_out=mask)
    torch.cuda.synchronize()
    ref = O.moe_step(x, w, acc if mode == "eat" else None, None, prm)
    border = PT.borderline(ref.routing, prm)
    err = PT.row_rel_err(_y_host(y), ref.y)[~border]
    assert (err <= (PT.TOL_Y_BF16 if shape.bf16 else PT.TOL_Y_F32)).all()
    if mode == "eat" and not border.any():
        n, pt, cs = lay.accounts_host()
        np.testing.assert_array_equal(n, ref.acc[0])
        np.testing.assert_allclose(pt, ref.acc[1], rtol=PT.TOL_P_TOTAL, atol=1e-6)


@pytest.mark.parametrize("case", ["finegrained", "qwen3", "qwen3_e256"])
def test_route_zero_input_takes_lowest_indices(case):
    # x = 0: every logit is 0, p is uniform; EAT with empty accounts has no
    # candidate and takes expert 0; Top-K takes experts 0..K-1 (word 0 only,
    # the other words stay 0).
    c = SMALL[case]
    for mode, expect in (("eat", 1), ("topk", (1 << 8) - 1)):
        shape, w, lay, prm = _layer(c, mode)
        x = torch.zeros(5, c["d"], dtype=torch.bfloat16, device="cuda")
        mask, k, gate, prob = lay.route(x)
        torch.cuda.synchronize()
        assert PT.masks_to_list(mask) == [expect] * 5
        np.testing.assert_allclose(prob.cpu().numpy(), 1.0 / c["E"], rtol=1e-6)


# ------------------------------------------------------------------ forward --

@pytest.mark.parametrize("case", ["tiny", "mixtral", "finegrained", "shared", "shared_split"] + WIDE_E)
@pytest.mark.parametrize("mode", ["eat", "topk", "topp"])
@pytest.mark.parametrize("T", [1, 33, 200])
def test_forward_parity(case, mode, T):
    c = SMALL[case]
    shape, w, lay, prm = _layer(c, mode)
    x = _x_host(shape, T, c["d"], seed=100 + T)
    acc = make_accounts(c["E"], seed=7 + T, c_scale=0.05)
    if mode == "eat":
        lay.load_accounts(*acc)
    mask = lay.mask_tensor(T)
    load = torch.empty(c["E"], dtype=torch.int32, device="cuda")
    y = lay.forward(_x_dev(x), mask_out=mask, load_out=load)
    torch.cuda.synchronize()
    ref = O.moe_step(x, w, acc if mode == "eat" else None, None, prm)
    border = PT.borderline(ref.routing, prm)
    gm = PT.masks_to_list(mask)
    bad = [t for t in range(T) if not border[t] and gm[t] != ref.routing.masks[t]]
    err = PT.row_rel_err(_y_host(y), ref.y)
    tol = PT.TOL_Y_BF16 if shape.bf16 else PT.TOL_Y_F32
    ok = ~border
    PT.report(f"forward {case} {mode} T={T}", borderline=int(border.sum()), mask_mismatch=len(bad),
              max_rel_y=f"{err[ok].max() if ok.any() else 0:.2e}")
    assert not bad
    assert (err[ok] <= tol).all()
    exp_load = [sum((m >> e) & 1 for m in gm) for e in range(c["E"])]
    assert load.cpu().numpy().tolist() == exp_load
    n, pt, cs = lay.accounts_host()
    if mode == "eat" and not border.any():
        np.testing.assert_array_equal(n, ref.acc[0])
        np.testing.assert_allclose(pt, ref.acc[1], rtol=PT.TOL_P_TOTAL, atol=1e-6)
        tol_c = PT.TOL_C_BF16 if shape.bf16 else PT.TOL_C_F32
        np.testing.assert_allclose(cs, ref.acc[2], rtol=tol_c, atol=1e-6)
    elif mode != "eat":
        assert (n == 0).all() and (pt == 0).all() and (cs == 0).all()


# degenerate configurations: one expert (fp32 and bf16, the smallest d and
# F), a cap equal to the expert count, Top-P with p = 1
DEGENERATE = {
    "one_expert_f32": (dict(shape="tiny", d=64, F=64, E=1, Fs=0), dict(K=1)),
    "one_expert_bf16": (dict(shape="mixtral", d=64, F=64, E=1, Fs=0), dict(K=1)),
    "cap_equals_e": (dict(shape="tiny", d=128, F=256, E=8, Fs=0), dict(K=8)),
    "cap_equals_e_bf16": (dict(shape="finegrained", d=256, F=256, E=64, Fs=0), dict(K=64)),
    "top_p_one": (dict(shape="tiny", d=128, F=256, E=8, Fs=0), dict(top_p=1.0)),
}


@pytest.mark.parametrize("name", list(DEGENERATE))
@pytest.mark.parametrize("mode", ["eat", "topk", "topp"])
@pytest.mark.parametrize("T", [1, 37])
def test_forward_degenerate_shapes(name, mode, T):
    c, kw = DEGENERATE[name]
    shape, w, lay, prm = _layer(c, mode, **kw)
    x = _x_host(shape, T, c["d"], seed=300 + T)
    acc = make_accounts(c["E"], seed=13 + T, c_scale=0.05)
    if mode == "eat":
        lay.load_accounts(*acc)
    mask = lay.mask_tensor(T)
    y = lay.forward(_x_dev(x), mask_out=mask)
    torch.cuda.synchronize()
    ref = O.moe_step(x, w, acc if mode == "eat" else None, None, prm)
    border = PT.borderline(ref.routing, prm)
    gm = PT.masks_to_list(mask)
    bad = [t for t in range(T) if not border[t] and gm[t] != ref.routing.masks[t]]
    err = PT.row_rel_err(_y_host(y), ref.y)
    ok = ~border
    PT.report(f"degenerate {name} {mode} T={T}", borderline=int(border.sum()), mask_mismatch=len(bad),
              max_rel_y=f"{err[ok].max() if ok.any() else 0:.2e}")
    assert not bad
    assert (err[ok] <= (PT.TOL_Y_BF16 if shape.bf16 else PT.TOL_Y_F32)).all()
    if c["E"] == 1:
        assert gm == [1] * T                  # every mode keeps the only expert
    if mode == "topp":
        # borderline Top-P tokens (p = 1 makes every token one) have several
        # correct answers: the mask must still be a prefix of the token's
        # descending-p order whose sum reaches p (to the band)
        for t in np.flatnonzero(border):
            pt_row = ref.routing.p[t]
            order = np.argsort(-pt_row, kind="stable")
            k = bin(gm[t]).count("1")
            assert sum(1 << int(i) for i in order[:k]) == gm[t], t
            assert pt_row[order[:k]].sum() >= prm.top_p - PT.EPS_B, t
    n, pt, cs = lay.accounts_host()
    if mode == "eat" and not border.any():
        np.testing.assert_array_equal(n, ref.acc[0])
        np.testing.assert_allclose(pt, ref.acc[1], rtol=PT.TOL_P_TOTAL, atol=1e-6)
        np.testing.assert_allclose(cs, ref.acc[2], rtol=PT.TOL_C_BF16 if shape.bf16 else PT.TOL_C_F32, atol=1e-6)
    lay.close()


# capped Top-P (top_p_cap): p = 0.9 so that the nucleus usually outgrows the
# cap; caps of 1, one within a mask word and one spanning words (E = 200)
@pytest.mark.parametrize("case,cap", [("tiny", 1), ("tiny", 3), ("finegrained", 3), ("finegrained", 8),
                                      ("qwen3", 5), ("qwen3_e200", 70)])
@pytest.mark.parametrize("T", [1, 37])
def test_forward_parity_topp_cap(case, cap, T):
    c = SMALL[case]
    shape, w, lay, prm = _layer(c, "topp", top_p=0.9, top_p_cap=cap)
    x = _x_host(shape, T, c["d"], seed=500 + T)
    mask = lay.mask_tensor(T)
    y = lay.forward(_x_dev(x), mask_out=mask)
    torch.cuda.synchronize()
    ref = O.moe_step(x, w, None, None, prm)
    border = PT.borderline(ref.routing, prm)
    gm = PT.masks_to_list(mask)
    bad = [t for t in range(T) if not border[t] and gm[t] != ref.routing.masks[t]]
    err = PT.row_rel_err(_y_host(y), ref.y)
    ok = ~border
    capped = int((ref.routing.k == cap).sum())
    PT.report(f"top-p cap {case} cap={cap} T={T}", borderline=int(border.sum()), mask_mismatch=len(bad),
              at_cap=capped, max_rel_y=f"{err[ok].max() if ok.any() else 0:.2e}")
    assert not bad
    assert all(bin(m).count("1") <= cap for m in gm)
    # borderline tokens (near-equal probabilities decide the order) must still
    # be valid capped nuclei: the selected experts outweigh the others (to the
    # band), and the prefix stops at the cap or once its sum reaches p
    for t in np.flatnonzero(border):
        pr = ref.routing.p[t]
        sel = np.array([(gm[t] >> e) & 1 for e in range(c["E"])], dtype=bool)
        assert sel.any(), t
        if (~sel).any():
            assert pr[sel].min() >= pr[~sel].max() - PT.EPS_B, t
        assert sel.sum() == cap or pr[sel].sum() >= prm.top_p - PT.EPS_B, t
    assert (err[ok] <= (PT.TOL_Y_BF16 if shape.bf16 else PT.TOL_Y_F32)).all()
    lay.close()


# every EAT hyper-parameter away from the paper's value (both sides get the
# same set), so a constant written into a kernel instead of its parameter
# shows; with a perplexity trend and two steps from zero accounts (the first
# step selects fewer than K experts for most of these sets, the EMA's alpha
# acts on the second step's accounts)
HYPER = [
    dict(beta=0.25, w1=0.5, w2=0.2, w3=0.3, alpha1=0.8, alpha2=0.4, kappa1=0.45, kappa2=0.55,
         ppl_up=1.5, ppl_down=0.75, q_lo=0.2, q_hi=0.8, alpha=0.7, eps=1e-6),
    dict(beta=0.9, w1=0.1, w2=0.6, w3=0.3, alpha1=0.2, alpha2=2.0, kappa1=1.0, kappa2=0.0,
         ppl_up=1.05, ppl_down=0.95, q_lo=0.0, q_hi=1.0, alpha=0.3, eps=1e-4),
]


@pytest.mark.parametrize("case", ["tiny", "finegrained", "qwen3"])
@pytest.mark.parametrize("hp", range(len(HYPER)))
def test_forward_parity_hyperparameters(case, hp):
    c = SMALL[case]
    shape = SHAPES[c["shape"]]
    kw = HYPER[hp]
    w = make_layer_weights(shape, E=c["E"], d=c["d"], F=c["F"], F_shared=c["Fs"])
    dt = L.EAT_BF16 if shape.bf16 else L.EAT_F32
    inv_t = 1.5
    p = L.eat_params_default(mode=L.EAT_MODE_EAT, E=c["E"], d_model=c["d"], d_ffn=c["F"], top_k=shape.K,
                             inv_temperature=inv_t, act_dtype=dt, expert_dtype=dt, **kw)
    lay = EatLayer(p, 64, to_device(w))
    prm = O.Params(mode=O.MODE_EAT, K=shape.K, inv_temp=inv_t, **kw)
    T = 37
    # zero accounts: the first step's importance is (1 - beta) p, so the
    # threshold parameters decide how many experts (fewer than K) survive
    acc = O.zero_accounts(c["E"])
    lay.load_accounts(*acc)
    for step in range(2):
        x = _x_host(shape, T, c["d"], seed=600 + 10 * hp + step)
        trend = make_trend(T, seed=700 + step)
        mask = lay.mask_tensor(T)
        y = lay.forward(_x_dev(x), trend=torch.from_numpy(trend).cuda(), mask_out=mask)
        torch.cuda.synchronize()
        ref = O.moe_step(x, w, acc, trend, prm)
        border = PT.borderline(ref.routing, prm)
        gm = PT.masks_to_list(mask)
        bad = [t for t in range(T) if not border[t] and gm[t] != ref.routing.masks[t]]
        err = PT.row_rel_err(_y_host(y), ref.y)
        ok = ~border
        PT.report(f"hyper-parameters {hp} {case} step {step}", borderline=int(border.sum()),
                  mask_mismatch=len(bad), mean_k=f"{np.mean(ref.routing.k):.2f}",
                  max_rel_y=f"{err[ok].max() if ok.any() else 0:.2e}")
        assert not bad
        assert (err[ok] <= (PT.TOL_Y_BF16 if shape.bf16 else PT.TOL_Y_F32)).all()
        n, pt, cs = lay.accounts_host()
        if border.any():
            break                           # the accounts may then differ legitimately
        np.testing.assert_array_equal(n, ref.acc[0])
        np.testing.assert_allclose(pt, ref.acc[1], rtol=PT.TOL_P_TOTAL, atol=1e-6)
        np.testing.assert_allclose(cs, ref.acc[2], rtol=PT.TOL_C_BF16 if shape.bf16 else PT.TOL_C_F32, atol=1e-6)
        acc = ref.acc
    lay.close()


def test_forward_ppl_trend_and_share_reading():
    c = SMALL["finegrained"]
    T = 64
    shape, w, lay, prm = _layer(c, "eat", cs_mode=1)
    x = _x_host(shape, T, c["d"], seed=5)
    trend = make_trend(T, seed=9)
    acc = make_accounts(c["E"], seed=11)
    lay.load_accounts(*acc)
    mask = torch.empty(T, dtype=torch.int64, device="cuda")
    y = lay.forward(_x_dev(x), trend=torch.from_numpy(trend).cuda(), mask_out=mask)
    torch.cuda.synchronize()
    ref = O.moe_step(x, w, acc, trend, prm)
    border = PT.borderline(ref.routing, prm)
    gm = PT.masks_to_list(mask)
    assert all(border[t] or gm[t] == ref.routing.masks[t] for t in range(T))
    err = PT.row_rel_err(_y_host(y), ref.y)
    assert (err[~border] <= PT.TOL_Y_BF16).all()


# ------------------------------------------------------- properties of runs --

def test_deterministic_and_permutation_equivariant():
    c = SMALL["mixtral"]
    T = 48
    shape, w, lay, prm = _layer(c, "eat")
    x = _x_host(shape, T, c["d"], seed=3)
    acc = make_accounts(c["E"], seed=4, c_scale=0.05)
    outs = []
    for _ in range(2):
        lay.load_accounts(*acc)
        y = lay.forward(_x_dev(x))
        torch.cuda.synchronize()
        outs.append((y.cpu().clone(), lay.accounts_host()))
    assert torch.equal(outs[0][0].view(torch.int16), outs[1][0].view(torch.int16))
    for a, b in zip(outs[0][1], outs[1][1]):
        np.testing.assert_array_equal(a, b)
    perm = np.random.default_rng(0).permutation(T)
    lay.load_accounts(*acc)
    yp = lay.forward(_x_dev(x[perm]))
    torch.cuda.synchronize()
    assert torch.equal(yp.cpu().view(torch.int16), outs[0][0][perm].view(torch.int16))
    n, pt, cs = lay.accounts_host()
    np.testing.assert_array_equal(n, outs[0][1][0])
    np.testing.assert_allclose(pt, outs[0][1][1], rtol=1e-6)
    np.testing.assert_allclose(cs, outs[0][1][2], rtol=1e-6)


def test_resume_from_saved_accounts():
    c = SMALL["tiny"]
    shape = SHAPES["tiny"]
    xs = HiddenStream(shape, 32, seed=21, d=c["d"]).steps(16)
    _, _, full, _ = _layer(c, "eat")
    ys_full = []
    for s in range(16):
        ys_full.append(full.forward(_x_dev(xs[s])).cpu())
    torch.cuda.synchronize()
    _, _, a, _ = _layer(c, "eat")
    for s in range(8):
        a.forward(_x_dev(xs[s]))
    saved = [t.clone() for t in (a.n, a.p_total, a.c_s)]
    _, _, b, _ = _layer(c, "eat")
    b.load_accounts(*[t.cpu() for t in saved])
    for s in range(8, 16):
        yb = b.forward(_x_dev(xs[s])).cpu()
        assert torch.equal(yb, ys_full[s])
    for u, v in zip((b.n, b.p_total, b.c_s), (full.n, full.p_total, full.c_s)):
        assert torch.equal(u.cpu(), v.cpu())


def test_reset_accounts_zeroes_state():
    c = SMALL["tiny"]
    _, _, lay, _ = _layer(c, "eat")
    lay.load_accounts(*make_accounts(8, seed=1))
    lay.reset_accounts()
    torch.cuda.synchronize()
    n, p, cs = lay.accounts_host()
    assert (n == 0).all() and (p == 0).all() and (cs == 0).all()


def test_trajectory_tiny_matches_oracle():
    """16 decode steps of the fp32 tiny layer, both sides from zero accounts.
    Masks must agree at every step up to the first borderline token (after
    it the two trajectories may legitimately part); the first divergent step
    is reported."""
    c = SMALL["tiny"]
    shape, w, lay, prm = _layer(c, "eat")
    xs = HiddenStream(shape, 32, d=c["d"]).steps(16)
    acc = O.zero_accounts(8)
    mask = torch.empty(32, dtype=torch.int64, device="cuda")
    ks = []
    for s in range(16):
        y = lay.forward(_x_dev(xs[s]), mask_out=mask)
        torch.cuda.synchronize()
        ref = O.moe_step(xs[s], w, acc, None, prm)
        border = PT.borderline(ref.routing, prm)
        if border.any():
            PT.report("trajectory tiny", first_borderline_step=s)
            return
        assert PT.masks_to_list(mask) == ref.routing.masks, f"step {s}"
        assert (PT.row_rel_err(_y_host(y), ref.y) <= PT.TOL_Y_F32).all()
        n, pt, cs = lay.accounts_host()
        np.testing.assert_array_equal(n, ref.acc[0])
        np.testing.assert_allclose(cs, ref.acc[2], rtol=PT.TOL_C_F32, atol=1e-6)
        ks.append(float(np.mean(ref.routing.k)))
        acc = ref.acc
    PT.report("trajectory tiny", steps=16, mean_k=f"{np.mean(ks):.3f}")


# ------------------------------------------------------------- full sizes --

@pytest.fixture(scope="module")
def mixtral_full():
    shape = SHAPES["mixtral"]
    return shape, make_layer_weights(shape)


@pytest.mark.parametrize("mode", ["topk", "eat"])
def test_full_mixtral_decode_sampled(mixtral_full, mode):
    """Mixtral-shaped layer at full size (d=4096, E=8, F=14336), decode batch
    64: routing of every token against the oracle, outputs of 6 sampled
    tokens (the oracle computes them one expert at a time)."""
    shape, w = mixtral_full
    T = 64
    p = L.eat_params_default(mode=MODES[mode], E=8, d_model=4096, d_ffn=14336, top_k=2,
                             inv_temperature=shape.inv_temp)
    lay = EatLayer(p, T, to_device(w))
    prm = PT.oracle_params(shape, MODES[mode])
    x = HiddenStream(shape, T).next()
    mask = torch.empty(T, dtype=torch.int64, device="cuda")
    y = lay.forward(_x_dev(x), mask_out=mask)
    torch.cuda.synchronize()
    r = O.route(x, w["w_router"], O.zero_accounts(8), None, prm)
    border = PT.borderline(r, prm)
    gm = PT.masks_to_list(mask)
    assert all(border[t] or gm[t] == r.masks[t] for t in range(T))
    sample = [t for t in (0, 9, 21, 38, 50, 63) if not border[t]]
    lo = O.layer_outputs(x, w, r, prm, tokens=sample)
    err = PT.row_rel_err(_y_host(y)[sample], lo.y[sample])
    PT.report(f"full mixtral {mode}", borderline=int(border.sum()), max_rel_y=f"{err.max():.2e}")
    assert (err <= PT.TOL_Y_BF16).all()
    lay.close()
    del lay
    torch.cuda.empty_cache()


@pytest.mark.parametrize("mode", ["topk", "topp", "eat"])
@pytest.mark.parametrize("T,prefill", [(256, False), (4096, True)])
def test_full_finegrained_sampled(mode, T, prefill):
    shape = SHAPES["finegrained"]
    w = make_layer_weights(shape)
    p = L.eat_params_default(mode=MODES[mode], E=64, d_model=2048, d_ffn=1024, top_k=8, top_p=0.6)
    lay = EatLayer(p, T, to_device(w))
    prm = PT.oracle_params(shape, MODES[mode])
    x = make_prefill(shape) if prefill else HiddenStream(shape, T).next()
    acc = make_accounts(64, seed=T, c_scale=0.05)
    if mode == "eat":
        lay.load_accounts(*acc)
    mask = torch.empty(T, dtype=torch.int64, device="cuda")
    y = lay.forward(_x_dev(x), mask_out=mask)
    torch.cuda.synchronize()
    r = O.route(x, w["w_router"], acc, None, prm)
    border = PT.borderline(r, prm)
    gm = PT.masks_to_list(mask)
    bad = [t for t in range(T) if not border[t] and gm[t] != r.masks[t]]
    rng = np.random.default_rng(T)
    sample = [int(t) for t in rng.choice(T, 24, replace=False) if not border[t]]
    lo = O.layer_outputs(x, w, r, prm, tokens=sample)
    err = PT.row_rel_err(_y_host(y)[sample], lo.y[sample])
    PT.report(f"full finegrained {mode} T={T}", borderline=int(border.sum()), mask_mismatch=len(bad),
              max_rel_y=f"{err.max():.2e}", mean_k=f"{np.mean(r.k):.3f}")
    assert not bad
    assert (err <= PT.TOL_Y_BF16).all()
    if mode == "eat" and not border.any():
        lo_all = O.layer_outputs(x, w, r, prm) if T <= 256 else None
        if lo_all is not None:
            ref_acc = O.account_update(acc, r.masks, r.p, lo_all.norms, prm)
            n, pt, cs = lay.accounts_host()
            np.testing.assert_array_equal(n, ref_acc[0])
            np.testing.assert_allclose(cs, ref_acc[2], rtol=PT.TOL_C_BF16, atol=1e-6)


@pytest.mark.parametrize("mode", ["topk", "topp", "eat"])
@pytest.mark.parametrize("T,prefill", [(64, False), (4096, True)])
def test_full_qwen3_sampled(mode, T, prefill):
    """Qwen3-30B-A3B-shaped layer at full size (d=2048, E=128, F=768, K=8):
    two mask words per token; decode batch 64 and a 4096-token prefill."""
    shape = SHAPES["qwen3"]
    w = make_layer_weights(shape)
    p = L.eat_params_default(mode=MODES[mode], E=128, d_model=2048, d_ffn=768, top_k=8, top_p=0.6)
    lay = EatLayer(p, T, to_device(w))
    prm = PT.oracle_params(shape, MODES[mode])
    x = make_prefill(shape) if prefill else HiddenStream(shape, T).next()
    acc = make_accounts(128, seed=T, c_scale=0.05)
    if mode == "eat":
        lay.load_accounts(*acc)
    mask = lay.mask_tensor(T)
    assert mask.shape == (T, 2)
    y = lay.forward(_x_dev(x), mask_out=mask)
    torch.cuda.synchronize()
    r = O.route(x, w["w_router"], acc, None, prm)
    border = PT.borderline(r, prm)
    gm = PT.masks_to_list(mask)
    bad = [t for t in range(T) if not border[t] and gm[t] != r.masks[t]]
    rng = np.random.default_rng(T)
    sample = [int(t) for t in rng.choice(T, 16, replace=False) if not border[t]]
    lo = O.layer_outputs(x, w, r, prm, tokens=sample)
    err = PT.row_rel_err(_y_host(y)[sample], lo.y[sample])
    PT.report(f"full qwen3 {mode} T={T}", borderline=int(border.sum()), mask_mismatch=len(bad),
              max_rel_y=f"{err.max():.2e}", mean_k=f"{np.mean(r.k):.3f}",
              upper_word_tokens=sum(1 for m in gm if m >> 64))
    assert not bad
    assert (err <= PT.TOL_Y_BF16).all()
    lay.close()
    del lay
    torch.cuda.empty_cache()


@pytest.mark.parametrize("T", [128, 8192])
def test_full_shared_sampled(T):
    shape = SHAPES["shared"]
    w = make_layer_weights(shape)
    p = L.eat_params_default(mode=L.EAT_MODE_TOPK, E=60, d_model=2048, d_ffn=1408, top_k=4,
                             d_shared=5632)
    lay = EatLayer(p, T, to_device(w))
    prm = PT.oracle_params(shape, O.MODE_TOPK, shared=True)
    x = make_prefill(shape) if T == 8192 else HiddenStream(shape, T).next()
    mask = torch.empty(T, dtype=torch.int64, device="cuda")
    y = lay.forward(_x_dev(x), mask_out=mask)
    torch.cuda.synchronize()
    r = O.route(x, w["w_router"], None, None, prm)
    border = PT.borderline(r, prm)
    gm = PT.masks_to_list(mask)
    assert all(border[t] or gm[t] == r.masks[t] for t in range(T))
    sample = [int(t) for t in np.random.default_rng(1).choice(T, 16, replace=False) if not border[t]]
    lo = O.layer_outputs(x, w, r, prm, tokens=sample)
    err = PT.row_rel_err(_y_host(y)[sample], lo.y[sample])
    PT.report(f"full shared T={T}", borderline=int(border.sum()), max_rel_y=f"{err.max():.2e}")
    assert (err <= PT.TOL_Y_BF16).all()


# --------------------------------------------- prefill-sized (tile kernels) --

TILE_CASES = {
    # 1024-1500 tokens over 8 experts, K=2: 256-375 rows per expert, so the
    # wide tiles run with partly filled token quarters and ragged tails
    "mixtral_tiles": dict(shape="mixtral", d=512, F=768, E=8, Fs=0),
    # shared expert of width 384 over 600 tokens goes through the wide tiles
    # (two full 256-token tiles and an 88-token half-height one)
    "shared_tiles": dict(shape="shared", d=256, F=192, E=60, Fs=384),
    # 2048-3000 tokens over 8 experts, K=2: 512-750 rows per expert, full
    # 256-token tiles plus ragged last ones
    "mixtral_wide": dict(shape="mixtral", d=512, F=768, E=8, Fs=0),
    # 4096-4500 tokens over 128 experts, K=8: ~256-280 rows per expert on
    # average, two mask words, 128 expert segments in the tile table
    "qwen3_wide": dict(shape="qwen3", d=256, F=256, E=128, Fs=0),
}


@pytest.mark.parametrize("mode", ["eat", "topk", "topp"])
@pytest.mark.parametrize("case,T", [("mixtral_tiles", 1024), ("mixtral_tiles", 1500), ("shared_tiles", 600),
                                    ("mixtral_wide", 2048), ("mixtral_wide", 3000),
                                    ("qwen3_wide", 4096), ("qwen3_wide", 4500)])
def test_forward_parity_prefill_tiles(case, T, mode):
    c = TILE_CASES[case]
    shape, w, lay, prm = _layer(c, mode, max_tokens=T)
    x = make_prefill(shape, tokens=T, seqs=4, d=c["d"])
    acc = make_accounts(c["E"], seed=T, c_scale=0.05)
    if mode == "eat":
        lay.load_accounts(*acc)
    mask = lay.mask_tensor(T)
    y = lay.forward(_x_dev(x), mask_out=mask)
    torch.cuda.synchronize()
    ref = O.moe_step(x, w, acc if mode == "eat" else None, None, prm)
    border = PT.borderline(ref.routing, prm)
    gm = PT.masks_to_list(mask)
    bad = [t for t in range(T) if not border[t] and gm[t] != ref.routing.masks[t]]
    err = PT.row_rel_err(_y_host(y), ref.y)
    ok = ~border
    PT.report(f"tiles {case} {mode} T={T}", borderline=int(border.sum()), mask_mismatch=len(bad),
              max_rel_y=f"{err[ok].max():.2e}")
    assert not bad
    assert (err[ok] <= PT.TOL_Y_BF16).all()
    if mode == "eat" and not border.any():
        n, pt, cs = lay.accounts_host()
        np.testing.assert_array_equal(n, ref.acc[0])
        np.testing.assert_allclose(cs, ref.acc[2], rtol=PT.TOL_C_BF16, atol=1e-6)
