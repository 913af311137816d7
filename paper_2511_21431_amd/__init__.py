"""MI355X-native chunked MoE expert layer (MemFine's per-GPU hot path).

The compute lives in libmemfine.so (hand-written gfx950 HIP kernels behind
the C ABI of include/memfine.h); this package only builds and binds it.
"""
from ._lib import (BF16, CHUNK_EXPERTS, CHUNK_TOKENS, ERR_SCRATCH, F32, NOALLOC_SCRATCH_BYTES, PASS_BWD, PASS_FWD, TILE_128, TILE_256, TILE_256_REG,  # noqa: F401
                   TILE_AUTO, MemfineError, TorchAllocator, lib, make_model, make_shape,
                   memfine_activation_memory, memfine_count, memfine_dispatch,
                   memfine_get_launch_options, memfine_mact_select, memfine_mact_thresholds,
                   memfine_moe_bwd, memfine_moe_fwd, memfine_moe_fwd_noalloc, memfine_plan, memfine_pool_high_water,
                   memfine_profile_begin, memfine_profile_end, memfine_router_bwd,
                   memfine_router_fwd, memfine_set_launch_options, memfine_static_memory,
                   memfine_status_str, memfine_workspace_bytes, memfine_workspace_held,
                   memfine_workspace_trim)
