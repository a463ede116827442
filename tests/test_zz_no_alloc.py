"""The allocation-free forward (eat_moe_forward_noalloc) against
eat_moe_forward on the same inputs and account state.

Both run the same kernels; only where the intermediates live differs (the
library's fixed device array against the caller's workspace), so outputs,
masks, expert loads and the account update must be bit-identical.  Each case
makes two calls in a row, the second with fewer tokens and other inputs, so
the second runs over what the first left in the shared array.  A call that
needs more than the array holds is rejected before anything is enqueued.
"""
import numpy as np
import pytest
import torch

from paper_2609_33614_amd import _lib as L
from paper_2609_33614_amd.layer import EatLayer, pack_weights, to_device
from workload import SHAPES, HiddenStream, make_accounts, make_layer_weights

pytestmark = pytest.mark.gpu

CASES = {
    # name: (shape, d, F, E, F_shared, mode, T1, T2, packed)
    "mixtral_eat": ("mixtral", 512, 768, 8, 0, "eat", 64, 20, False),
    "finegrained_topk": ("finegrained", 256, 256, 64, 0, "topk", 200, 33, False),
    "qwen3_eat": ("qwen3", 256, 256, 128, 0, "eat", 64, 5, False),
    "shared_topp": ("shared", 256, 192, 60, 1024, "topp", 128, 17, False),
    "mixtral_full_eat": ("mixtral", 4096, 14336, 8, 0, "eat", 64, 8, True),
}


def _noalloc(lay, x, y, mask, load):
    w = lay.w
    L.eat_moe_forward_noalloc(lay.handle, x, x.shape[0], w["w_router"], w["w1"], w["w3"], w["w2"], w.get("ws1"),
                              w.get("ws3"), w.get("ws2"), lay.acc, None, y, mask, load)


@pytest.mark.parametrize("name", list(CASES))
def test_noalloc_matches_workspace_forward(name):
    shape_name, d, F, E, Fs, mode, T1, T2, packed = CASES[name]
    shape = SHAPES[shape_name]
    w = to_device(make_layer_weights(shape, E=E, d=d, F=F, F_shared=Fs))
    if packed:
        w = pack_weights(w)
    p = L.eat_params_default(mode=L.MODES[mode], E=E, d_model=d, d_ffn=F, top_k=shape.K,
                             top_p=shape.top_p or 0.6, inv_temperature=shape.inv_temp, d_shared=Fs,
                             weight_layout=L.EAT_LAYOUT_PACKED if packed else L.EAT_LAYOUT_ROWS)
    ref, lay = EatLayer(p, T1, w), EatLayer(p, T1, w)
    acc = make_accounts(E, seed=E, c_scale=0.05)
    if mode == "eat":
        ref.load_accounts(*acc)
        lay.load_accounts(*acc)
    hs = HiddenStream(shape, T1, d=d)
    for step, T in enumerate((T1, T2)):
        assert L.eat_workspace_size(lay.handle, T) <= L.EAT_NOALLOC_SCRATCH_BYTES
        x = torch.from_numpy(hs.next()[:T]).view(torch.bfloat16).cuda()
        m_ref, m_new = lay.mask_tensor(T), lay.mask_tensor(T)
        l_ref = torch.empty(E, dtype=torch.int32, device="cuda")
        l_new = torch.full((E,), -1, dtype=torch.int32, device="cuda")
        y_ref = ref.forward(x, mask_out=m_ref, load_out=l_ref)
        y_new = torch.full_like(x, float("nan"))
        _noalloc(lay, x, y_new, m_new, l_new)
        torch.cuda.synchronize()
        print(f"[noalloc] {name} call {step}: T={T} workspace={L.eat_workspace_size(lay.handle, T) >> 20} MiB",
              flush=True)
        assert torch.equal(y_new.view(torch.int16), y_ref.view(torch.int16)), f"call {step}: outputs differ"
        assert torch.equal(m_new, m_ref), f"call {step}: masks differ"
        assert torch.equal(l_new, l_ref), f"call {step}: expert loads differ"
        for a, b in zip(lay.accounts_host(), ref.accounts_host()):
            np.testing.assert_array_equal(a, b)
    ref.close()
    lay.close()
    del w
    torch.cuda.empty_cache()


def test_noalloc_rejects_calls_beyond_the_scratch_limit():
    shape = SHAPES["finegrained"]
    T = 256
    w = to_device(make_layer_weights(shape))
    p = L.eat_params_default(mode=L.EAT_MODE_EAT, E=64, d_model=2048, d_ffn=1024, top_k=8)
    lay = EatLayer(p, T, w)
    assert L.eat_workspace_size(lay.handle, T) > L.EAT_NOALLOC_SCRATCH_BYTES
    x = torch.from_numpy(HiddenStream(shape, T).next()).view(torch.bfloat16).cuda()
    y = torch.zeros_like(x)
    with pytest.raises(L.EatError) as ei:
        _noalloc(lay, x, y, None, None)
    torch.cuda.synchronize()
    assert ei.value.status == L.EAT_ERR_SCRATCH_LIMIT
    assert not y.view(torch.int16).any()            # nothing was enqueued
    assert (lay.accounts_host()[0] == 0).all()
    lay.close()
