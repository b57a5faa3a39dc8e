"""Pins of the lazy-checkpoint oracle (Sec. 5.2) against what the paper and the
mathematics fix: a hand-enumerated scenario (tests/golden/lazy_checkpoint.json),
the definition of a gather as indexing of the pool's (block, slot) rows, the
oracle's independently pinned sequence gather, and the invariant the mechanism
exists for -- a peer's attention is unchanged by checkpoint, overwrite and
restore. The last test plants mistakes in the oracle and checks that a pin
catches each one."""

import json
import os

import numpy as np
import pytest

from oracle import checkpoint as ck
from oracle import paged_attention as pa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLDEN = os.path.join(ROOT, "tests", "golden", "lazy_checkpoint.json")


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


def _random(rng, shape, dtype):
    """Random finite values: fp32 normals, or bf16 bit patterns with the top
    exponent bit clear (|x| < 2, never Inf or NaN)."""
    if dtype == "bf16":
        return rng.integers(0, 1 << 16, size=shape, dtype=np.uint16) & np.uint16(0xBFFF)
    return rng.standard_normal(shape).astype(np.float32)


def _random_pool(rng, num_blocks, hkv, d, dtype):
    return _random(rng, (num_blocks, hkv, 16, d), dtype)


def _rows_by_indexing(pool, ids):
    """The gather's definition with numpy indexing: the pool viewed as
    [slot id][Hkv][D] rows."""
    nb, hkv, bs, d = pool.shape
    flat = pool.transpose(0, 2, 1, 3).reshape(nb * bs, hkv, d)
    ids = np.asarray(ids, dtype=np.int64)
    ok = (ids >= 0) & (ids < nb * bs)
    out = np.zeros((len(ids), hkv, d), dtype=pool.dtype)
    out[ok] = flat[ids[ok]]
    return out


# --- the hand-enumerated scenario ---------------------------------------------

def _scenario_tables(g):
    """Sequences 0 = B (RT), 1 = a (BE) as block tables padded to 2 entries."""
    B, a = g["before"]["B"], g["before"]["a"]
    tables = np.full((2, 2), -1, dtype=np.int32)
    tables[0, :len(B["block_table"])] = B["block_table"]
    tables[1, :len(a["block_table"])] = a["block_table"]
    tables[1, 1] = 0          # never read: a's context stays inside entry 0
    dirs = np.array([B["dir"], a["dir"]], dtype=np.int8)
    ctx = np.array([B["ctx"], a["ctx"]], dtype=np.int32)
    return tables, dirs, ctx


def test_scenario_layout_matches_fixture():
    g = _golden()
    tables, dirs, ctx = _scenario_tables(g)
    blocks, slots = pa.physical_location(tables, dirs, 1, np.arange(ctx[1]))
    assert [[p, s] for p, (b, s) in enumerate(zip(blocks, slots)) if b == 3] == g["before"]["a"]["in_block_3"]
    blocks, slots = pa.physical_location(tables, dirs, 0, np.arange(16, ctx[0]))
    assert [[p, s] for p, s in zip(range(16, ctx[0]), slots)] == g["before"]["B"]["tail_in_block_3"]
    assert set(blocks.tolist()) == {3}
    # block 3 is full before the write: every slot owned exactly once
    counts = pa.slot_owner_counts(tables, dirs, ctx, g["num_blocks"])
    assert counts[3].tolist() == [1] * 16


def test_overwritten_peer_tokens_match_fixture():
    g = _golden()
    tables, dirs, ctx = _scenario_tables(g)
    w = g["write"]
    victims = ck.overwritten_peer_tokens(tables, dirs, ctx, 0, w["positions"])
    assert [["a" if s == 1 else "B", p, b, sl] for s, p, b, sl in victims] == g["checkpoint"]
    ids = ck.slot_ids([v[2] for v in victims], [v[3] for v in victims])
    assert ids.tolist() == g["checkpoint_slot_ids"]
    # the writer's new slots are exactly the fixture's
    b, s = pa.physical_location(tables, dirs, 0, np.array(w["positions"]))
    assert [[int(x), int(y)] for x, y in zip(b, s)] == w["block_slot"]


def test_no_victims_while_slots_remain():
    # a block with free slots: the writer's new positions land on empty slots
    tables = np.array([[1, 3], [3, 0]], dtype=np.int32)
    dirs = np.array([1, -1], dtype=np.int8)
    ctx = np.array([18, 10], dtype=np.int32)          # B uses slots 0-1, a slots 15..6
    assert ck.overwritten_peer_tokens(tables, dirs, ctx, 0, [18, 19, 20, 21]) == []   # slots 2-5 are free
    assert len(ck.overwritten_peer_tokens(tables, dirs, ctx, 0, [18, 19, 20, 21, 22])) == 1   # slot 6 is a's


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_checkpoint_overwrite_restore_keeps_peer_attention(dtype):
    """Sec. 5.2's point: after the peer's tokens are checkpointed, overwritten
    by the writer and restored into a fresh block, the peer attends to exactly
    the tokens it had (bit-identical fp64 result); without the checkpoint its
    attention would change."""
    g = _golden()
    rng = np.random.default_rng(11)
    hkv, hq, d = 2, 4, 128
    nb = g["num_blocks"]
    tables, dirs, ctx = _scenario_tables(g)
    k_pool = _random_pool(rng, nb, hkv, d, dtype)
    v_pool = _random_pool(rng, nb, hkv, d, dtype)
    q2 = _random(rng, (2, hq, d), dtype)      # row 1 is a's query
    before = pa.decode(q2, k_pool, v_pool, tables, dirs, ctx, dtype, seqs=[1])[1]

    # 1. checkpoint the victims (gather to "CPU memory")
    w = g["write"]
    victims = ck.overwritten_peer_tokens(tables, dirs, ctx, 0, w["positions"])
    ids = ck.slot_ids([v[2] for v in victims], [v[3] for v in victims])
    saved_k, saved_v = ck.kv_gather(k_pool, ids), ck.kv_gather(v_pool, ids)

    # 2. the writer stores its new tokens over them
    n = len(w["positions"])
    k_new = _random(rng, (n, hkv, d), dtype)
    v_new = _random(rng, (n, hkv, d), dtype)
    k1, v1 = pa.kv_write(k_pool, v_pool, k_new, v_new, tables, dirs,
                         np.array([w["positions"][0], 0]), np.array([0, n, n]))
    ctx_after = ctx.copy()
    ctx_after[0] += n
    damaged = pa.decode(q2, k1, v1, tables, dirs, ctx_after, dtype, seqs=[1])[1]
    assert not np.array_equal(damaged, before)

    # 3. restore: a's table entry 0 moves to a fresh block; its surviving tokens
    #    are moved there and the checkpointed ones are swapped back in
    r = g["restore"]
    new_tables = tables.copy()
    new_tables[1, r["table_entry"]] = r["new_block"]
    lost = {v[1] for v in victims}
    keep_pos = [p for p in range(int(ctx[1])) if p not in lost]
    ob, os_ = pa.physical_location(tables, dirs, 1, np.array(keep_pos))
    nb_, ns_ = pa.physical_location(new_tables, dirs, 1, np.array(keep_pos))
    moved_k = ck.kv_gather(k1, ck.slot_ids(ob, os_))
    moved_v = ck.kv_gather(v1, ck.slot_ids(ob, os_))
    k2 = ck.kv_scatter(k1, moved_k, ck.slot_ids(nb_, ns_))
    v2 = ck.kv_scatter(v1, moved_v, ck.slot_ids(nb_, ns_))
    rb, rs = pa.physical_location(new_tables, dirs, 1, np.array([v[1] for v in victims]))
    k2 = ck.kv_scatter(k2, saved_k, ck.slot_ids(rb, rs))
    v2 = ck.kv_scatter(v2, saved_v, ck.slot_ids(rb, rs))
    # the new locations are the fixture's
    allb, alls = pa.physical_location(new_tables, dirs, 1, np.arange(int(ctx[1])))
    assert [[p, int(b), int(s)] for p, (b, s) in enumerate(zip(allb, alls))] == r["position_to_block_slot"]
    after = pa.decode(q2, k2, v2, new_tables, dirs, ctx_after, dtype, seqs=[1])[1]
    assert np.array_equal(after, before)
    # and the writer sees its own tokens, not the peer's
    wrote = pa.gather_kv(k2, new_tables, dirs, 0, int(ctx_after[0]))[16:]
    assert np.array_equal(wrote[-n:], k_new)


# --- gather and scatter as data movement ----------------------------------------

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gather_is_indexing_of_slot_rows(dtype):
    rng = np.random.default_rng(5)
    pool = _random_pool(rng, 9, 3, 8, dtype)
    ids = rng.permutation(9 * 16)[:50].astype(np.int64)
    ids[[3, 17]] = [-1, 9 * 16]                       # outside the pool: zero rows
    got = ck.kv_gather(pool, ids)
    assert got.dtype == pool.dtype
    assert np.array_equal(got.view(np.uint8), _rows_by_indexing(pool, ids).view(np.uint8))
    assert not got[3].any() and not got[17].any()


def test_gather_of_a_sequence_is_its_cache():
    """The slot ids of a sequence's positions gather exactly its cached tensors
    (the oracle's sequence gather is pinned by the layout fixture and dense
    attention)."""
    rng = np.random.default_rng(6)
    pool = _random_pool(rng, 12, 2, 8, "f32")
    tables = np.array([[4, 7, 2], [7, 1, 0]], dtype=np.int32)
    dirs = np.array([1, -1], dtype=np.int8)
    for s, ctx in ((0, 40), (1, 25)):
        b, sl = pa.physical_location(tables, dirs, s, np.arange(ctx))
        assert np.array_equal(ck.kv_gather(pool, ck.slot_ids(b, sl)), pa.gather_kv(pool, tables, dirs, s, ctx))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_scatter_then_gather_round_trip(dtype):
    rng = np.random.default_rng(7)
    pool = _random_pool(rng, 6, 2, 8, dtype)
    ids = rng.permutation(6 * 16)[:30].astype(np.int64)
    ids[5] = -3                                         # skipped
    rows = _random(rng, (30, 2, 8), dtype)
    out = ck.kv_scatter(pool, rows, ids)
    back = ck.kv_gather(out, ids)
    ok = ids >= 0
    assert np.array_equal(back[ok].view(np.uint8), rows[ok].view(np.uint8))
    # every slot not named keeps its bytes
    touched = np.zeros(6 * 16, dtype=bool)
    touched[ids[ok]] = True
    flat_in = pool.transpose(0, 2, 1, 3).reshape(96, 2, 8)
    flat_out = out.transpose(0, 2, 1, 3).reshape(96, 2, 8)
    assert np.array_equal(flat_in[~touched].view(np.uint8), flat_out[~touched].view(np.uint8))
    assert np.array_equal(pool, ck.kv_scatter(pool, rows[:0], ids[:0]))   # empty list: nothing moves


def test_scatter_rejects_repeated_slot():
    pool = np.zeros((2, 1, 16, 4), dtype=np.float32)
    with pytest.raises(ValueError):
        ck.kv_scatter(pool, np.ones((2, 1, 4), np.float32), [3, 3])


# --- planted mistakes -------------------------------------------------------------

def test_pins_catch_planted_mistakes(monkeypatch):
    """Each plausible slip in the checkpoint oracle breaks some pin above."""
    real_gather, real_victims = ck.kv_gather, ck.overwritten_peer_tokens

    def gather_wrong_slot(pool, ids):       # slot counted from the other end
        nb, hkv, bs, d = pool.shape
        ids = np.asarray(ids, dtype=np.int64)
        return real_gather(pool, (ids // bs) * bs + (bs - 1 - ids % bs))

    def victims_off_by_one(tables, dirs, ctx, writer, pos):   # misses the last new position
        return real_victims(tables, dirs, ctx, writer, list(pos)[:-1])

    for name, fake in (("kv_gather", gather_wrong_slot), ("overwritten_peer_tokens", victims_off_by_one)):
        monkeypatch.setattr(ck, name, fake)
        failed = 0
        for t in (test_overwritten_peer_tokens_match_fixture, test_gather_of_a_sequence_is_its_cache,
                  lambda: test_checkpoint_overwrite_restore_keeps_peer_attention("f32")):
            try:
                t()
            except AssertionError:
                failed += 1
        assert failed > 0, name
        monkeypatch.setattr(ck, name, real_gather if name == "kv_gather" else real_victims)
