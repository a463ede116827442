"""EAT (Expert Account Tracker) MoE-layer forward for MI355X (gfx950).

The compute lives in libeat.so (hand-written HIP kernels behind the C ABI
of include/eat.h); this package only builds and binds it.
"""
from ._lib import (  # noqa: F401
    EAT_BF16, EAT_F32, EAT_MODE_EAT, EAT_MODE_TOPK, EAT_MODE_TOPP, EatError, LIB_PATH, MODES,
    accounts, eat_accounts_t, eat_create, eat_destroy, eat_moe_forward, eat_moe_forward_profiled, eat_params_default,
    eat_params_t, eat_reset_accounts, eat_route, eat_route_workspace_size, eat_stack_forward, eat_stack_layer_t,
    eat_stack_workspace_size, eat_status_string, eat_workspace_size, load, stack_layers, eat_ppl_workspace_size,
    eat_ppl_reset, eat_ppl_trend, EAT_LAYOUT_PACKED, EAT_LAYOUT_ROWS, eat_pack_weights, mask_words,
    eat_moe_forward_noalloc, EAT_NOALLOC_SCRATCH_BYTES,
)
