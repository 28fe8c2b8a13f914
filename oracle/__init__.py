"""fp64 CPU oracle for chunk-wise causal attention.

TEST INFRASTRUCTURE ONLY: used by tests/, the smoke check and the benchmark's
CPU-baseline leg.  The HIP library never imports, links or calls it."""
from .chunk_attention import (  # noqa: F401
    attention,
    attention_bwd,
    attention_bwd_delta,
    attention_bwd_keys,
    brute_force,
    count_visible_pairs,
    frame_mask,
    key_chunks,
    kv_cache_append,
    query_chunks,
    ring_slot,
    ring_step,
    softmax_weights,
    visibility_mask,
)
from .one_step import one_step_update, target_velocity  # noqa: F401
from .tiles import axis_weights, tile_axis, tile_blend, tile_gather  # noqa: F401
