"""CPU fp64 oracle for one paged-attention step over a mixed RT/BE batch.

TEST INFRASTRUCTURE ONLY. This module is the slow, obviously-correct statement of
what the HIP path computes. Only the test suite, the smoke check and the CPU
baseline leg of the benchmark import it; the product path never does, and it
shares no code with the HIP kernels, their host library or their binding.

What it follows (the paper: "Efficient LLM Serving on Hybrid Real-time and
Best-effort Requests", arXiv 2504.09590):

* Bidirectional block layout, Sec. 5.1 (Block Structure): GPU KV memory is a
  pool of blocks of slots; the KV of an RT request fills a block's slots from
  the left end to the right end, the KV of a BE request fills them from the
  right end to the left end, and one block may hold one of each.
* Exclusive view, Sec. 5.2 (Block Management, lazy checkpointing): while free
  slots remain, each of the two requests treats a shared block as its own, so
  block i of a request's block table holds that request's logical positions
  [16 i, 16 i + 16), in its own direction.
* Direction table, Sec. 6 (Implementation): a binary flag, shaped like the
  block tables, says whether the slots of a block are walked from the left or
  from the right. Here +1 means left-to-right and -1 right-to-left; a flag per
  sequence is broadcast over that sequence's block-table row.
* Mixed batch, Sec. 6: prefill requests are concatenated along the token axis
  and their shapes kept in a length table; decode requests follow. Attention
  over cached context is softmax(q k^T * scale) v per query head (Sec. 2.1
  describes decode as reusing the cached keys and values of earlier tokens;
  Sec. 4.1 prices attention by the L^n x L^a score matrix).

Readings where the paper is silent: the softmax scale is 1/sqrt(D); query
head h reads KV head h // (Hq // Hkv) (consecutive query heads share a KV
head); a decode sequence's context length counts the token written this step;
the causal diagonal is inclusive; a decode sequence with no context yields a
zero output row.

Every floating-point computation here runs in float64. bf16 inputs arrive as
uint16 bit patterns and are widened exactly (bf16 -> fp32 -> fp64 is exact).
"""

from __future__ import annotations

import numpy as np

BLOCK_SIZE = 16  # slots per block; the paper's systems all use 16 (Sec. 7.1)


# --------------------------------------------------------------------------
# exact widening of the two storage dtypes
# --------------------------------------------------------------------------

def widen(x: np.ndarray, dtype: str) -> np.ndarray:
    """Return x as float64. dtype 'bf16' means x holds bf16 bit patterns (uint16)."""
    if dtype == "bf16":
        bits = np.asarray(x).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


# --------------------------------------------------------------------------
# the bidirectional slot mapping (Sec. 5.1, Sec. 5.2 exclusive view, Sec. 6)
# --------------------------------------------------------------------------

def slot_in_block(p, direction):
    """Slot holding logical position p inside its block.

    Left-to-right (+1, the RT direction of Sec. 5.1): offset p mod 16 counted
    from the left end. Right-to-left (-1, the BE direction): the same offset
    counted from the right end.
    """
    offset = np.asarray(p) % BLOCK_SIZE
    direction = np.asarray(direction)
    if np.any((direction != 1) & (direction != -1)):
        raise ValueError("direction flags must be +1 or -1")
    return np.where(direction == 1, offset, BLOCK_SIZE - 1 - offset)


def _direction_of(dir_flags: np.ndarray, s: int, block_index):
    """Direction of block-table entry block_index of sequence s.

    Accepts a per-sequence flag vector [S] or a per-entry table [S][max_blocks]
    (the paper's form, Sec. 6)."""
    dir_flags = np.asarray(dir_flags)
    if dir_flags.ndim == 1:
        return np.broadcast_to(dir_flags[s], np.shape(block_index))
    return dir_flags[s][block_index]


def physical_location(block_tables, dir_flags, s: int, positions):
    """(block id, slot) of each logical position of sequence s."""
    positions = np.asarray(positions, dtype=np.int64)
    block_index = positions // BLOCK_SIZE
    blocks = np.asarray(block_tables)[s][block_index].astype(np.int64)
    slots = slot_in_block(positions, _direction_of(dir_flags, s, block_index))
    return blocks, slots


def gather_kv(pool: np.ndarray, block_tables, dir_flags, s: int, ctx: int) -> np.ndarray:
    """Sequence s's cached tensors in logical order: [ctx, Hkv, D].

    pool has the layout [num_blocks][Hkv][16][D]. Only the (block, slot) pairs
    that hold positions 0..ctx-1 are read; every other slot is ignored."""
    blocks, slots = physical_location(block_tables, dir_flags, s, np.arange(ctx))
    return pool[blocks, :, slots, :]


# --------------------------------------------------------------------------
# plain softmax attention (Sec. 2.1, Sec. 4.1)
# --------------------------------------------------------------------------

def softmax_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                      limits: np.ndarray, scale: float) -> np.ndarray:
    """Attention of n query rows over one sequence's cached keys/values.

    q: [n, Hq, D]; k, v: [ctx, Hkv, D]; limits[j]: row j sees keys 0..limits[j]-1.
    Query head h reads KV head h // (Hq // Hkv). Returns [n, Hq, D] float64.
    A row with limit 0 has no keys and returns zeros."""
    n, hq, d = q.shape
    ctx, hkv = k.shape[0], k.shape[1]
    group = hq // hkv
    limits = np.asarray(limits, dtype=np.int64)
    visible = np.arange(ctx)[None, :] < limits[:, None]       # [n, ctx]
    has_keys = limits > 0
    out = np.zeros((n, hq, d), dtype=np.float64)
    for h in range(hq):
        kh = k[:, h // group, :]                                # [ctx, D]
        vh = v[:, h // group, :]
        scores = (q[:, h, :] @ kh.T) * scale                    # [n, ctx]
        row_max = np.where(visible, scores, -np.inf).max(axis=1, initial=-np.inf)
        shift = np.where(has_keys, row_max, 0.0)[:, None]
        w = np.where(visible, np.exp(np.where(visible, scores, 0.0) - shift), 0.0)
        total = w.sum(axis=1)
        out[has_keys, h, :] = (w[has_keys] @ vh) / total[has_keys, None]
    return out


def default_scale(head_dim: int) -> float:
    return 1.0 / np.sqrt(head_dim)


# --------------------------------------------------------------------------
# the three operations of the step
# --------------------------------------------------------------------------

def kv_write(k_pool, v_pool, k_new, v_new, block_tables, dir_flags, pos0, cu_new):
    """Store each new token's K/V in the slot its sequence's direction dictates.

    Token t of sequence s (t in [cu_new[s], cu_new[s+1])) has logical position
    pos0[s] + (t - cu_new[s]); its [Hkv][D] rows go to that position's (block,
    slot) (Sec. 5.1 layout, Sec. 5.2 exclusive view). Returns new pools; every
    other byte is copied unchanged. Pure data movement: dtype-agnostic."""
    k_out = np.array(k_pool, copy=True)
    v_out = np.array(v_pool, copy=True)
    cu_new = np.asarray(cu_new)
    for s in range(len(cu_new) - 1):
        first, last = int(cu_new[s]), int(cu_new[s + 1])
        if last == first:
            continue
        positions = int(pos0[s]) + np.arange(last - first)
        blocks, slots = physical_location(block_tables, dir_flags, s, positions)
        for i, t in enumerate(range(first, last)):
            k_out[blocks[i], :, slots[i], :] = k_new[t]
            v_out[blocks[i], :, slots[i], :] = v_new[t]
    return k_out, v_out


def decode(q, k_pool, v_pool, block_tables, dir_flags, ctx_lens, dtype: str,
           scale: float | None = None, seqs=None) -> np.ndarray:
    """One decode query row per sequence over its whole cached context.

    q: [S][Hq][D]; returns [S][Hq][D] float64 (rows outside `seqs` stay zero
    when a subset is requested)."""
    qf = widen(q, dtype)
    kf = widen(k_pool, dtype)
    vf = widen(v_pool, dtype)
    S, hq, d = qf.shape
    scale = default_scale(d) if scale is None else scale
    out = np.zeros((S, hq, d), dtype=np.float64)
    for s in (range(S) if seqs is None else seqs):
        ctx = int(ctx_lens[s])
        k = gather_kv(kf, block_tables, dir_flags, s, ctx)
        v = gather_kv(vf, block_tables, dir_flags, s, ctx)
        out[s] = softmax_attention(qf[s:s + 1], k, v, np.array([ctx]), scale)[0]
    return out


def prefill_chunk(q, cu_q, k_pool, v_pool, block_tables, dir_flags, ctx_lens,
                  dtype: str, scale: float | None = None, seqs=None) -> np.ndarray:
    """Causal attention of each sequence's new rows on top of its prior context.

    Rows of sequence s are q[cu_q[s]:cu_q[s+1]] (the length table of Sec. 6);
    with n = cu_q[s+1] - cu_q[s] and c0 = ctx_lens[s] - n, row j sits at
    position c0 + j and sees keys 0..c0 + j (diagonal inclusive)."""
    qf = widen(q, dtype)
    kf = widen(k_pool, dtype)
    vf = widen(v_pool, dtype)
    T, hq, d = qf.shape
    scale = default_scale(d) if scale is None else scale
    out = np.zeros((T, hq, d), dtype=np.float64)
    cu_q = np.asarray(cu_q)
    for s in (range(len(cu_q) - 1) if seqs is None else seqs):
        first, last = int(cu_q[s]), int(cu_q[s + 1])
        n = last - first
        if n == 0:
            continue
        ctx = int(ctx_lens[s])
        c0 = ctx - n
        if c0 < 0:
            raise ValueError(f"sequence {s}: {n} new rows exceed context {ctx}")
        k = gather_kv(kf, block_tables, dir_flags, s, ctx)
        v = gather_kv(vf, block_tables, dir_flags, s, ctx)
        limits = c0 + np.arange(n) + 1
        out[first:last] = softmax_attention(qf[first:last], k, v, limits, scale)
    return out


# --------------------------------------------------------------------------
# batch consistency (Sec. 5.2: two sequences never own the same slot)
# --------------------------------------------------------------------------

def owned_slots(block_tables, dir_flags, ctx_lens):
    """Set of (block, slot) pairs holding some sequence's valid position, with
    the owner. Raises if two positions land on one slot."""
    owner = {}
    for s in range(len(ctx_lens)):
        blocks, slots = physical_location(block_tables, dir_flags, s, np.arange(int(ctx_lens[s])))
        for p, (b, sl) in enumerate(zip(blocks.tolist(), slots.tolist())):
            key = (b, sl)
            if key in owner:
                raise ValueError(f"slot {key} owned by {owner[key]} and ({s}, {p})")
            owner[key] = (s, p)
    return owner


def slot_owner_counts(block_tables, dir_flags, ctx_lens, num_blocks: int) -> np.ndarray:
    """[num_blocks][16] count of valid positions mapped to each slot; a
    consistent batch has no entry above 1."""
    counts = np.zeros((num_blocks, BLOCK_SIZE), dtype=np.int32)
    for s in range(len(ctx_lens)):
        blocks, slots = physical_location(block_tables, dir_flags, s, np.arange(int(ctx_lens[s])))
        np.add.at(counts, (blocks, slots), 1)
    return counts
