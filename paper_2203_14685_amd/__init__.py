"""MI355X-native MoE gate / layout-transform hot path (HetuMoE, arXiv 2203.14685).

The compute lives in libhetumoe.so (hand-written HIP kernels for gfx950, C ABI
in include/hetumoe.h); this package is its thin Python binding.
"""

from .binding import (  # noqa: F401
    EXPORTED,
    LIB_PATH,
    MOE_BF16,
    MOE_F32,
    MOE_GATE_HASH,
    MOE_GATE_HTOPK,
    MOE_GATE_KTOP1,
    MOE_GATE_TOPK,
    MoeError,
    GateBwdParams,
    GateParams,
    Layout,
    combine,
    combine_bwd,
    dispatch,
    dispatch_bwd,
    gate,
    gate_bwd,
    gate_bwd_params,
    gate_params,
    load,
    moe_combine,
    moe_combine_bwd,
    moe_dispatch,
    moe_dispatch_bwd,
    moe_gate,
    moe_gate_bwd,
    moe_gate_bwd_workspace_size,
    moe_gate_workspace_size,
    moe_hash_balanced_table,
)
