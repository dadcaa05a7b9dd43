"""True-tail hybrid-state update on MI355X (gfx950).

The HIP library libtailupdate.so (built from csrc/ by `build.py`) implements the
update of a hybrid recurrent-attention context (paper Section 4.1, Eq. 2-3): KV
compaction, rotary append at the true tail, causal GQA attention over surviving
+ new KV, and the gated delta-rule continuation from the carried state.
It also continues the recurrent layers' short convolution from its carried state,
and provides the slot-preserving and tail-and-relocate placements the paper compares
(Section 5.2) together with the relocation of stored keys, and the attention
diagnostics of Section 5.3 (probe distributions, group masses, total variation).
`binding` is the ctypes layer over its C ABI (include/tailupdate.h).
"""
from .binding import (  # noqa: F401
    Context,
    LayerIO,
    StackUpdate,
    TailUpdateError,
    attention_group_mass,
    attention_probe,
    attention_tv_distance,
    attn_params,
    commit_tail,
    compact_kv,
    compact_kv_noalloc,
    delta_params,
    delta_rule_continue,
    new_vt_cache,
    vt_cache_bytes,
    workspace_faults,
    lib,
    profile_collect,
    profile_enable,
    refresh_vt_cache,
    relocate_keys,
    short_conv_continue,
    short_conv_continue_batch,
    tail_prefill_attention,
    update_layer_stack,
    TU_FAULT_POSITIONS,
    TU_FAULT_RANGE,
    TU_FAULT_WAIT,
    TU_LAYER_ATTN,
    TU_LAYER_DELTA,
    TU_PLACE_RELOCATE,
    TU_PLACE_SLOT,
    TU_PLACE_TAIL,
)
