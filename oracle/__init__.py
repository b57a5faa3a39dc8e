"""CPU oracle for the bidirectional paged-attention step (test infrastructure only).

Imported by the test suite, the smoke check and the benchmark's CPU baseline leg;
never by the product path.
"""
from .paged_attention import (  # noqa: F401
    BLOCK_SIZE, widen, slot_in_block, physical_location, gather_kv,
    softmax_attention, default_scale, kv_write, decode, prefill_chunk, owned_slots,
    slot_owner_counts,
)
from .checkpoint import (  # noqa: F401
    slot_ids, kv_gather, kv_scatter, overwritten_peer_tokens,
)
