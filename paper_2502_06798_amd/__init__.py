"""apc: approximate-cache prompt matching on MI355X (gfx950).

The per-batch step of prompt-aware scheduling for diffusion serving with
approximate caching: nearest cached prompts (cosine top-k), optimal skip
level, capacity-constrained placement on model instances, and the gather of
the cached latents.  The compute lives in hand-written HIP kernels behind the
C ABI of include/apc.h; this package is its thin Python binding plus the
seeded synthetic workload generator (synth).
"""
from .binding import (APC_BF16, APC_E4M3, APC_F16, APC_F32, APC_MAX_INST, APC_MAX_K,
                      APC_MAX_LEVELS, ApcError, Cache, apc_assign, apc_assign_load_aware, apc_assign_planned,
                      apc_assign_routed, apc_build_cache,
                      apc_cache_row_factors, apc_destroy_cache, apc_gather_latents,
                      apc_gather_latents_at_level,
                      apc_last_error, apc_level_histogram, apc_match_batch, apc_match_batch_static, apc_match_workspace,
                      apc_merge_shards, apc_quantize_rows, apc_resident_best, apc_route_plan,
                      apc_row_factors, apc_set_kernel_events, apc_status_str, apc_validate_rows, load,
                      workspace_tensor)
from .pipeline import MatchStep

__all__ = ["APC_BF16", "APC_E4M3", "APC_F16", "APC_F32", "APC_MAX_INST", "APC_MAX_K",
           "APC_MAX_LEVELS", "ApcError", "Cache", "MatchStep", "apc_assign", "apc_assign_load_aware",
           "apc_assign_planned",
           "apc_assign_routed", "apc_build_cache",
           "apc_cache_row_factors", "apc_destroy_cache", "apc_gather_latents",
           "apc_gather_latents_at_level", "apc_last_error",
           "apc_level_histogram", "apc_match_batch", "apc_match_batch_static", "apc_match_workspace", "apc_merge_shards",
           "apc_quantize_rows", "apc_resident_best",
           "apc_route_plan", "apc_row_factors", "apc_set_kernel_events",
           "apc_status_str", "apc_validate_rows", "load",
           "workspace_tensor"]
