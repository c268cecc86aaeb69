"""FreqCache per-step hot path on AMD Instinct MI355X (gfx950).

Frequency-guided cacheable-token selection feeding a partial-recompute decoder
layer, as hand-written HIP behind a C ABI (include/freqcache.h).  This package
is the Python binding (argument marshalling only) plus the in-tree build step.
"""
from .freqcache import (  # noqa: F401
    Caps, Context, FcError, KVCache, LayerDesc, SelectOut, SelectParams, EXPORTS, COUNTS,
    SCALARS, FLAG_ALIGNED, FLAG_CAND, FLAG_FRESH, fc_cache_update, fc_cache_update_layers,
    fc_create, fc_cache_step, FC_ADVANCE_WINDOW, FC_REMAP, fc_debug, fc_destroy, fc_last_error,
    fc_layer_forward, fc_layer_forward_trail,
    fc_phase_correlate, fc_phase_correlate_rotation, fc_profile_enable, fc_profile_only,
    fc_profile_read, fc_select, fc_select_noalloc,
    fc_select_carry, fc_vit_block_forward, fc_vit_cache_update, fc_vit_merger_forward,
    MergerDesc, VitCache, VitDesc,
    select_state_bytes, select_state_alloc, fc_slot_map_init, slot_state_alloc,
    slot_state_bytes, fc_version, lib, token_grid)
