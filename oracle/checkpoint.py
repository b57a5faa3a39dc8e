"""CPU oracle for lazy checkpointing of shared blocks (test infrastructure only).

TEST INFRASTRUCTURE ONLY, like the rest of this package: the test suite and the
benchmark's CPU leg import it, the product path never does.

What it follows (Sec. 5.2, Block Management, "Lazy checkpointing"; Sec. 6 on
the fetch/store kernels and the separate streams):

* While a shared block still has empty slots, its RT and BE occupants each
  treat it as their own (the exclusive view). Once the slots run out, the
  occupant about to write a new token may take a slot that still holds a
  token of its peer. Only those peer tokens are copied to CPU memory (the
  checkpoint), not the peer's whole cache, and the block is marked as
  preempted.
* When the peer is scheduled again, its checkpointed tokens are copied back
  to GPU memory.

Slots are named by one integer, slot id = block * 16 + slot. The two data
movements are a gather of the rows at a list of slot ids into a dense
[n][Hkv][D] buffer (the layout of a step's new tokens) and the scatter back.

Reading where the paper is silent: a restored token goes wherever the block
manager points the peer's table entry when it is scheduled again. The
scenario in the tests gives that entry a fresh block and moves the entry's
surviving tokens there too, so the peer's table keeps the exclusive view.
An id outside the pool reads as a zero row and is never written.
"""

from __future__ import annotations

import numpy as np

from .paged_attention import BLOCK_SIZE, physical_location


def slot_ids(blocks, slots) -> np.ndarray:
    """Slot ids (block * 16 + slot) of (block, slot) pairs."""
    return (np.asarray(blocks, dtype=np.int64) * BLOCK_SIZE + np.asarray(slots, dtype=np.int64)).astype(np.int32)


def kv_gather(pool: np.ndarray, ids) -> np.ndarray:
    """Rows of pool ([num_blocks][Hkv][16][D]) at the given slot ids, as
    [n][Hkv][D]. An id outside the pool yields a zero row. Pure data movement:
    the rows keep their bit patterns."""
    num_blocks, hkv, bs, d = pool.shape
    out = np.zeros((len(ids), hkv, d), dtype=pool.dtype)
    for i, sid in enumerate(np.asarray(ids, dtype=np.int64).tolist()):
        if 0 <= sid < num_blocks * bs:
            out[i] = pool[sid // bs, :, sid % bs, :]
    return out


def kv_scatter(pool: np.ndarray, rows: np.ndarray, ids) -> np.ndarray:
    """A copy of pool with rows[i] ([Hkv][D]) stored at slot id ids[i]. Ids
    outside the pool are skipped; the ids inside it must be distinct."""
    num_blocks, hkv, bs, d = pool.shape
    out = np.array(pool, copy=True)
    seen = set()
    for i, sid in enumerate(np.asarray(ids, dtype=np.int64).tolist()):
        if 0 <= sid < num_blocks * bs:
            if sid in seen:
                raise ValueError(f"slot id {sid} appears twice")
            seen.add(sid)
            out[sid // bs, :, sid % bs, :] = rows[i]
    return out


def overwritten_peer_tokens(block_tables, dir_flags, ctx_lens, writer: int, new_positions):
    """Tokens of other sequences held in the slots that sequence `writer`'s
    new positions map to (the tokens Sec. 5.2 checkpoints before the write).

    Returns a list of (sequence, position, block, slot), in sequence then
    position order."""
    wb, ws = physical_location(block_tables, dir_flags, writer, np.asarray(new_positions))
    taken = set(zip(wb.tolist(), ws.tolist()))
    victims = []
    for s in range(len(ctx_lens)):
        if s == writer:
            continue
        ctx = int(ctx_lens[s])
        if ctx == 0:
            continue
        blocks, slots = physical_location(block_tables, dir_flags, s, np.arange(ctx))
        for p, (b, sl) in enumerate(zip(blocks.tolist(), slots.tolist())):
            if (b, sl) in taken:
                victims.append((s, p, b, sl))
    return victims
