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


def _check_routing(name, r, prm, mask, gate, prob, k, shift=0.0):
    """Routing outputs against the oracle's: p within TOL_P; masks bit-exact
    outside the band (4x the observed |dp|), valid inside it; gates and
    expert counts of every token (the borderline ones from the GPU's
    validated choice).  Returns the routing with those choices adopted."""
    dp = float(np.abs(prob.cpu().numpy() - r.p).max())
    band = PT.band_for(dp)
    assert dp <= PT.TOL_P, f"{name}: router probabilities differ by {dp:.2e}"
    assert band <= PT.BAND_MAX
    gm = PT.masks_to_list(mask)
    border, ra = PT.compare_masks(name, gm, r, prm, band, shift)
    dg = float(np.abs(gate.cpu().numpy() - ra.g_norm).max())
    kk = k.cpu().numpy()
    PT.report(name, T=len(gm), band=f"{band:.1e}", borderline=int(border.sum()), max_dp=f"{dp:.2e}",
              max_dgate=f"{dg:.2e}", mean_k=f"{kk.mean():.3f}")
    assert dg <= PT.TOL_P
    assert (kk == ra.k).all()
    return border, ra


def _forward_check(name, lay, shape, x, w, prm, acc=None, trend=None, tokens=None, check_acc=True,
                   shift=0.0):
    """One layer forward through the C ABI against the oracle.

    Routing (eat_route on the same inputs and account state: the same
    kernels the forward runs) gives the observed |dp| and so the band; the
    forward's masks must equal the routing call's, match the oracle outside
    the band and be valid inside it; the layer output of every token (or of
    ``tokens``) is compared with the oracle's for the selection taken (the
    borderline tokens' validated choice adopted), and in EAT mode the
    account update (Sec. 3.2) with it.  Returns (adopted routing, the
    oracle's new accounts or None, the borderline flags)."""
    T = x.shape[0]
    E = prm_E = lay.params.E
    eat = prm.mode == O.MODE_EAT
    if eat:
        lay.load_accounts(*acc)
    xd = _x_dev(x)
    td = torch.from_numpy(trend).cuda() if trend is not None else None
    mask_r, k, gate, prob = lay.route(xd, td)
    mask = lay.mask_tensor(T)
    load = torch.empty(E, dtype=torch.int32, device="cuda")
    y = lay.forward(xd, trend=td, mask_out=mask, load_out=load)
    torch.cuda.synchronize()
    r = O.route(x, w["w_router"], acc if eat else None, trend, prm)
    assert PT.masks_to_list(mask) == PT.masks_to_list(mask_r), f"{name}: forward and routing masks differ"
    border, ra = _check_routing(name, r, prm, mask, gate, prob, k, shift)
    gm = PT.masks_to_list(mask)
    exp_load = [sum((m >> e) & 1 for m in gm) for e in range(prm_E)]
    assert load.cpu().numpy().tolist() == exp_load
    lo = O.layer_outputs(x, w, ra, prm, tokens=tokens)
    rows = np.arange(T) if tokens is None else np.array(sorted(set(int(t) for t in tokens)))
    err = PT.row_rel_err(_y_host(y)[rows], lo.y[rows])
    tol = PT.TOL_Y_BF16 if shape.bf16 else PT.TOL_Y_F32
    PT.report(name + " output", rows=len(rows), max_rel_y=f"{err.max():.2e}",
              borderline_rows=int(border[rows].sum()))
    assert (err <= tol).all(), f"{name}: output error {err.max():.2e}"
    n, pt, cs = lay.accounts_host()
    ref_acc = None
    if eat and check_acc and tokens is None:
        ref_acc = O.account_update(acc, ra.masks, ra.p, lo.norms, prm)
        np.testing.assert_array_equal(n, ref_acc[0])
        np.testing.assert_allclose(pt, ref_acc[1], rtol=PT.TOL_P_TOTAL, atol=1e-6)
        tol_c = PT.TOL_C_BF16 if shape.bf16 else PT.TOL_C_F32
        np.testing.assert_allclose(cs, ref_acc[2], rtol=tol_c, atol=1e-6)
    elif not eat:
        assert (n == 0).all() and (pt == 0).all() and (cs == 0).all()
    return ra, ref_acc, border


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
    gates, probabilities, and the forward's output and accounts)."""
    c = SMALL[case]
    T = 200
    scale = make_expert_scale(c["E"], seed=17)
    shape, w, lay, prm = _layer(c, mode, scale=scale)
    x = _x_host(shape, T, c["d"], seed=55)
    acc = make_accounts(c["E"], seed=3, c_scale=0.05)
    ra, _, _ = _forward_check(f"opd {case} {mode} T={T}", lay, shape, x, w, prm, acc=acc)
    # the scales change the selection of some tokens (the hook is live)
    plain = O.route(x, w["w_router"], acc, None, PT.oracle_params(shape, MODES[mode]))
    assert sum(a != b for a, b in zip(plain.masks, ra.masks)) > 0


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
    _forward_check(f"forward {case} {mode} T={T}", lay, shape, x, w, prm, acc=acc)


# larger decode-sized calls on the 64-expert layer: several 128-token tiles
# per expert, the slice counts the device picks for 256-513 tokens
@pytest.mark.parametrize("mode", ["eat", "topk", "topp"])
@pytest.mark.parametrize("T", [256, 512, 513])
def test_forward_parity_larger_decodes(mode, T):
    c = SMALL["finegrained"]
    shape, w, lay, prm = _layer(c, mode, max_tokens=T)
    x = _x_host(shape, T, c["d"], seed=400 + T)
    acc = make_accounts(c["E"], seed=T, c_scale=0.05)
    _forward_check(f"larger decode {mode} T={T}", lay, shape, x, w, prm, acc=acc)


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
    ra, _, _ = _forward_check(f"degenerate {name} {mode} T={T}", lay, shape, x, w, prm, acc=acc)
    if c["E"] == 1:
        assert ra.masks == [1] * T              # every mode keeps the only expert
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
    ra, _, _ = _forward_check(f"top-p cap {case} cap={cap} T={T}", lay, shape, x, w, prm)
    PT.report(f"top-p cap {case} cap={cap} T={T}", at_cap=int((ra.k == cap).sum()))
    assert all(bin(m).count("1") <= cap for m in ra.masks)
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
    # threshold parameters decide how many experts (fewer than K) survive;
    # the second step routes against the first step's update (injected)
    acc = O.zero_accounts(c["E"])
    for step in range(2):
        x = _x_host(shape, T, c["d"], seed=600 + 10 * hp + step)
        trend = make_trend(T, seed=700 + step)
        ra, acc, _ = _forward_check(f"hyper-parameters {hp} {case} step {step}", lay, shape, x, w, prm, acc=acc,
                                    trend=trend)
        PT.report(f"hyper-parameters {hp} {case} step {step}", mean_k=f"{np.mean(ra.k):.2f}")
    lay.close()


def test_forward_ppl_trend_and_share_reading():
    c = SMALL["finegrained"]
    T = 64
    shape, w, lay, prm = _layer(c, "eat", cs_mode=1)
    x = _x_host(shape, T, c["d"], seed=5)
    trend = make_trend(T, seed=9)
    acc = make_accounts(c["E"], seed=11)
    _forward_check("share reading with trends", lay, shape, x, w, prm, acc=acc, trend=trend)


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


@pytest.mark.parametrize("case", WIDE_E)
def test_reset_accounts_every_expert(case):
    """Sec. 3.2: the statistics start empty.  eat_reset_accounts must clear
    all E entries (here 100 to 256, several 64-expert groups), and a forward
    after it must equal the oracle's from zero accounts."""
    c = SMALL[case]
    E, T = c["E"], 37
    shape, w, lay, prm = _layer(c, "eat")
    g = np.random.default_rng(E)
    full = (g.integers(1, 500, E).astype(np.int64), g.uniform(0.5, 9.0, E).astype(np.float32),
            g.uniform(0.1, 2.0, E).astype(np.float32))
    lay.load_accounts(*full)
    x0 = _x_host(shape, T, c["d"], seed=900)
    lay.forward(_x_dev(x0))                       # a forward on the loaded history first
    torch.cuda.synchronize()
    assert (lay.accounts_host()[0] > 0).all()
    lay.reset_accounts()
    torch.cuda.synchronize()
    n, pt, cs = lay.accounts_host()
    PT.report(f"reset {case}", E=E, nonzero_after_reset=int((n != 0).sum() + (pt != 0).sum() + (cs != 0).sum()))
    assert (n == 0).all() and (pt == 0).all() and (cs == 0).all()
    # the forward after the reset routes as from zero accounts
    x1 = _x_host(shape, T, c["d"], seed=901)
    ra = O.route(x1, w["w_router"], O.zero_accounts(E), None, prm)
    mask = lay.mask_tensor(T)
    lay.forward(_x_dev(x1), mask_out=mask)
    torch.cuda.synchronize()
    gm = PT.masks_to_list(mask)
    border = PT.borderline(ra, prm)
    assert all(border[t] or gm[t] == ra.masks[t] for t in range(T))
    n, _, _ = lay.accounts_host()
    assert n.sum() == sum(bin(m).count("1") for m in gm)


# Free-running EAT decode from zero accounts: the GPU keeps its own account
# state; the oracle follows (the H rounding of the GPU's bf16 path modelled,
# reading R27), adopting the GPU's validated choice for every borderline
# token, so the two trajectories stay on one path and every step is checked
# in full.  The two account states differ only by rounding; that difference
# joins the band through its bound on the history score.  Reported: the
# first step with a borderline token (where an oracle running on its own
# could have left the GPU's path) and the largest account drift.
TRAJ = {
    "tiny": (dict(shape="tiny", d=128, F=256, E=8, Fs=0), 32, 16),
    "mixtral": (dict(shape="mixtral", d=512, F=768, E=8, Fs=0), 64, 32),
    "finegrained": (dict(shape="finegrained", d=256, F=256, E=64, Fs=0), 64, 32),
    "qwen3": (dict(shape="qwen3", d=256, F=256, E=128, Fs=0), 64, 24),
}


@pytest.mark.parametrize("case", list(TRAJ))
def test_trajectory_matches_oracle(case):
    c, B, steps = TRAJ[case]
    shape, w, lay, prm = _layer(c, "eat")
    prm.round_h = shape.bf16
    xs = HiddenStream(shape, B, d=c["d"]).steps(steps)
    acc = O.zero_accounts(c["E"])
    first, borders, drift, ks = None, 0, 0.0, []
    for s in range(steps):
        gpu_acc = lay.accounts_host()
        shift = PT.history_shift(gpu_acc, acc, prm)
        x = xs[s]
        xd = _x_dev(x)
        mask_r, k, gate, prob = lay.route(xd)
        mask = lay.mask_tensor(B)
        y = lay.forward(xd, mask_out=mask)
        torch.cuda.synchronize()
        r = O.route(x, w["w_router"], acc, None, prm)
        border, ra = _check_routing(f"trajectory {case} step {s}", r, prm, mask, gate, prob, k, shift)
        assert PT.masks_to_list(mask) == PT.masks_to_list(mask_r)
        lo = O.layer_outputs(x, w, ra, prm)
        err = PT.row_rel_err(_y_host(y), lo.y)
        assert (err <= (PT.TOL_Y_BF16 if shape.bf16 else PT.TOL_Y_F32)).all(), f"step {s}: {err.max():.2e}"
        acc = O.account_update(acc, ra.masks, ra.p, lo.norms, prm)
        n, pt, cs = lay.accounts_host()
        np.testing.assert_array_equal(n, acc[0])
        np.testing.assert_allclose(pt, acc[1], rtol=PT.TOL_P_TOTAL, atol=1e-6)
        np.testing.assert_allclose(cs, acc[2], rtol=PT.TOL_C_BF16 if shape.bf16 else PT.TOL_C_F32, atol=1e-6)
        drift = max(drift, float(np.max(np.abs(cs.astype(np.float64) - acc[2]) / np.maximum(np.abs(acc[2]), 1e-6))))
        if border.any() and first is None:
            first = s
        borders += int(border.sum())
        ks.append(float(np.mean(ra.k)))
    PT.report(f"trajectory {case}", steps=steps, tokens=B, first_borderline_step=first, borderline_tokens=borders,
              max_rel_c_drift=f"{drift:.1e}", mean_k=f"{np.mean(ks):.3f}")


# ------------------------------------------------------------- full sizes --

@pytest.fixture(scope="module")
def mixtral_full():
    shape = SHAPES["mixtral"]
    w = make_layer_weights(shape)
    return shape, w, PT.CachedWeights(w)


def test_full_mixtral_decode_topk(mixtral_full):
    """Mixtral-shaped layer at full size (d=4096, E=8, F=14336), decode
    batch 64, Top-K: every token's routing and output."""
    shape, w, wc = mixtral_full
    T = 64
    p = L.eat_params_default(mode=L.EAT_MODE_TOPK, E=8, d_model=4096, d_ffn=14336, top_k=2,
                             inv_temperature=shape.inv_temp)
    lay = EatLayer(p, T, to_device(w))
    prm = PT.oracle_params(shape, O.MODE_TOPK)
    _forward_check("full mixtral topk", lay, shape, HiddenStream(shape, T).next(), wc, prm)
    lay.close()
    del lay
    torch.cuda.empty_cache()


@pytest.mark.parametrize("layout", ["packed", "rows"])
def test_full_mixtral_decode_eat_timed_regime(mixtral_full, layout):
    """The benchmarked regime: the Mixtral-shaped layer at full size, decode
    batch 64, 8 EAT steps from zero accounts on the benchmark's inputs.  The
    oracle's account state is loaded before every step, so the GPU routes
    against exactly the state the oracle holds and the routing concentrates
    as in the benchmark (a few experts with 64-token tiles, the down
    projection in 8 slices); every token's mask and output and the account
    update are compared at every step."""
    from paper_2609_33614_amd.layer import pack_weights
    shape, w, wc = mixtral_full
    T = 64
    lay_w = to_device(w)
    if layout == "packed":
        lay_w = pack_weights(lay_w)
    p = L.eat_params_default(mode=L.EAT_MODE_EAT, E=8, d_model=4096, d_ffn=14336, top_k=2,
                             inv_temperature=shape.inv_temp,
                             weight_layout=L.EAT_LAYOUT_PACKED if layout == "packed" else L.EAT_LAYOUT_ROWS)
    lay = EatLayer(p, T, lay_w)
    prm = PT.oracle_params(shape, O.MODE_EAT)
    hs = HiddenStream(shape, T)
    acc = O.zero_accounts(8)
    unions = []
    for s in range(8):
        x = hs.next()
        ra, acc, _ = _forward_check(f"full mixtral eat {layout} step {s}", lay, shape, x, wc, prm, acc=acc)
        unions.append(bin(int(np.bitwise_or.reduce(np.array(ra.masks, dtype=object)))).count("1"))
    PT.report(f"full mixtral eat {layout}", experts_touched=unions)
    assert min(unions[2:]) < 8            # the history concentrates the steps' picks
    lay.close()
    del lay, lay_w
    torch.cuda.empty_cache()


@pytest.mark.parametrize("mode", ["topk", "topp", "eat"])
@pytest.mark.parametrize("T,prefill", [(256, False), (4096, True)])
def test_full_finegrained(mode, T, prefill):
    """Fine-grained layer at full size (d=2048, E=64, F=1024, K=8): decode
    batch 256 and the 4096-token prefill; every token's output and, in EAT
    mode, the account update."""
    shape = SHAPES["finegrained"]
    w = make_layer_weights(shape)
    p = L.eat_params_default(mode=MODES[mode], E=64, d_model=2048, d_ffn=1024, top_k=8, top_p=0.6)
    lay = EatLayer(p, T, to_device(w))
    prm = PT.oracle_params(shape, MODES[mode])
    x = make_prefill(shape) if prefill else HiddenStream(shape, T).next()
    acc = make_accounts(64, seed=T, c_scale=0.05)
    ra, _, _ = _forward_check(f"full finegrained {mode} T={T}", lay, shape, x, PT.CachedWeights(w), prm, acc=acc)
    PT.report(f"full finegrained {mode} T={T}", mean_k=f"{np.mean(ra.k):.3f}")
    lay.close()
    del lay
    torch.cuda.empty_cache()


@pytest.mark.parametrize("mode", ["topk", "topp", "eat"])
@pytest.mark.parametrize("T,prefill", [(64, False), (4096, True)])
def test_full_qwen3(mode, T, prefill):
    """Qwen3-30B-A3B-shaped layer at full size (d=2048, E=128, F=768, K=8):
    two mask words per token; decode batch 64 and a 4096-token prefill;
    every token's output and, in EAT mode, the account update of all 128
    experts."""
    shape = SHAPES["qwen3"]
    w = make_layer_weights(shape)
    p = L.eat_params_default(mode=MODES[mode], E=128, d_model=2048, d_ffn=768, top_k=8, top_p=0.6)
    lay = EatLayer(p, T, to_device(w))
    prm = PT.oracle_params(shape, MODES[mode])
    x = make_prefill(shape) if prefill else HiddenStream(shape, T).next()
    acc = make_accounts(128, seed=T, c_scale=0.05)
    ra, _, _ = _forward_check(f"full qwen3 {mode} T={T}", lay, shape, x, PT.CachedWeights(w), prm, acc=acc)
    PT.report(f"full qwen3 {mode} T={T}", mean_k=f"{np.mean(ra.k):.3f}",
              upper_word_tokens=sum(1 for m in ra.masks if m >> 64))
    lay.close()
    del lay
    torch.cuda.empty_cache()


@pytest.mark.parametrize("mode", ["topk", "topp", "eat"])
@pytest.mark.parametrize("T", [128, 8192])
def test_full_shared(mode, T):
    """Shared-expert layer at full size (60 experts of width 1408 + the
    always-on expert of width 5632, K=4): decode batch 128 (every token) and
    the 8192-token prefill (48 sampled tokens, and the EAT account update's
    N and P_total, which need no outputs)."""
    shape = SHAPES["shared"]
    w = make_layer_weights(shape)
    p = L.eat_params_default(mode=MODES[mode], E=60, d_model=2048, d_ffn=1408, top_k=4, top_p=0.6,
                             d_shared=5632)
    lay = EatLayer(p, T, to_device(w))
    prm = PT.oracle_params(shape, MODES[mode], shared=True)
    x = make_prefill(shape) if T == 8192 else HiddenStream(shape, T).next()
    acc = make_accounts(60, seed=T, c_scale=0.05)
    wc = PT.CachedWeights(w)
    if T == 8192:
        sample = [int(t) for t in np.random.default_rng(1).choice(T, 48, replace=False)]
        ra, _, _ = _forward_check(f"full shared {mode} T={T}", lay, shape, x, wc, prm, acc=acc, tokens=sample)
        if mode == "eat":
            n, pt, _ = lay.accounts_host()
            n_ref = acc[0] + np.array([sum((m >> e) & 1 for m in ra.masks) for e in range(60)])
            np.testing.assert_array_equal(n, n_ref)
            p_ref = [np.float32(np.float64(acc[1][e]) + sum(ra.p[t, e] for t in range(T) if (ra.masks[t] >> e) & 1))
                     for e in range(60)]
            np.testing.assert_allclose(pt, p_ref, rtol=PT.TOL_P_TOTAL, atol=1e-6)
    else:
        _forward_check(f"full shared {mode} T={T}", lay, shape, x, wc, prm, acc=acc)
    lay.close()
    del lay
    torch.cuda.empty_cache()


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
    _forward_check(f"tiles {case} {mode} T={T}", lay, shape, x, w, prm, acc=acc)
