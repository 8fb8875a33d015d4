"""Schedule-level shared-prefix attention for MI355X (gfx950).

The computation lives in the HIP library ``lib/libspr.so`` (C ABI in
``include/spr.h``); ``binding`` marshals torch tensors into it and
``group`` keeps one prompt group resident in HBM and runs the three-phase
schedule or the dense-recompute baseline through the binding.
"""
from .binding import (SprDims, SprError, make_dims, prefix_fwd, suffix_attn_fwd,
                      suffix_attn_bwd_accum, prefix_bwd, dense_recompute_baseline,
                      workspace_size, gkv_cache_zero, gkv_accumulate, profile_enable,
                      profile_reset, profile_query, profile_kernels, version)

__all__ = ["SprDims", "SprError", "make_dims", "prefix_fwd", "suffix_attn_fwd",
           "suffix_attn_bwd_accum", "prefix_bwd", "dense_recompute_baseline", "workspace_size",
           "gkv_cache_zero", "gkv_accumulate", "profile_enable", "profile_reset",
           "profile_query", "profile_kernels", "version"]
