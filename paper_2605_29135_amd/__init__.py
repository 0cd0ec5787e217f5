"""MoE decode step under a fixed HBM expert budget, for MI355X (gfx950).

The work runs in ``libmoe_budget.so`` (hand-written HIP kernels and a C++
residency runtime, C ABI in ``include/moe_budget.h``); :mod:`.binding` only
marshals torch device tensors into it.
"""
from .binding import (  # noqa: F401
    EVENT_HIT, EVENT_MISS, EVENT_PREFETCH, EVENT_HOST, MOE_SLOT_HOST, HostTier, MOE_ACCUMULATE, MOE_BF16, MOE_ROUTE_RMSNORM, MOE_F32, MOE_INT4G128, MOE_POLICY_LRU, MOE_POLICY_ROTARY, ExpertCache,
    MoeError, MoeStack, PinnedBuffer, header_symbols, lib, moe_combine, moe_expert_ffn_grouped, moe_expert_ffn_grouped_noalloc, moe_hbm_read_probe, moe_opt_fills, moe_opt_fills_flat,
    moe_ffn_workspace_bytes, moe_init, moe_prefill_grouped, moe_prefill_workspace_bytes, moe_route_topk,
    moe_sync_check, moe_attention_decode, moe_attention_workspace_bytes, key_cache_layout, key_cache_plain)
