"""MoE dispatch/combine hot path for one MI355X (gfx950).

The operator itself is the C ABI in include/moe.h, implemented by the HIP
kernels under csrc/ and built into libmoe.so; `moe` is its ctypes binding.
"""
from .moe import (  # noqa: F401
    EXPORTS, MOE_DTYPE_BF16, MOE_DTYPE_FP8_E4M3, MOE_PLAN_PARTS, MOE_POLICY_BALANCED,
    MOE_POLICY_BY_RANK, MOE_POLICY_DYNAMIC, MOE_POLICY_ROWS, MOE_POLICY_STATIC,
    MOE_STATUS_BAD_INDEX,
    MOE_STATUS_CAPACITY, MOE_STATUS_DUP_INDEX, DedupLayout, Layout, MoeError, Regions, lib,
    moe_combine, moe_combine_dedup, moe_combine_ex, moe_combine_local, moe_dispatch,
    moe_dispatch_dedup, moe_dispatch_ex, moe_expand, moe_expert_scale, moe_layout,
    moe_layout_dedup, moe_layout_dedup_workspace_bytes, moe_layout_fixed,
    moe_layout_workspace_bytes, moe_version)
