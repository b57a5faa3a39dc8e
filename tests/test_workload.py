"""The seeded generator emits the five workloads with the stated shapes,
length ranges, classes, directions and pool occupancies, and every batch it
emits is consistent (no slot owned twice)."""

import numpy as np
import pytest

import oracle
from paper_2504_09590_amd import workload as W

RANGES = {  # config: {class: (lo, hi)}
    1: {W.RT: (17, 300), W.BE: (17, 300)},
    2: {W.RT: (128, 2048), W.BE: (1024, 8192)},
    3: {W.RT: (512, 2048 + 512), W.BE: (512, 8192)},
    4: {W.RT: (256, 4096), W.BE: (2048, 16384)},
    5: {W.RT: (16, 32768), W.BE: (16, 32768)},
}
COUNTS = {1: (2, 2), 2: (16, 48), 3: (4, 128), 4: (32, 256), 5: (128, 384)}
HEADS = {1: (8, 8), 2: (32, 8), 3: (32, 8), 4: (64, 8), 5: (32, 8)}


@pytest.fixture(scope="module", params=[1, 2, 3, 4, 5])
def batch(request):
    return W.generate(request.param, with_pool=(request.param == 1))


def test_shapes_classes_and_directions(batch):
    c = batch.meta["config"]
    n_rt, n_be = COUNTS[c]
    assert (batch.cls == W.RT).sum() == n_rt and (batch.cls == W.BE).sum() == n_be
    assert np.all(batch.dir[batch.cls == W.RT] == 1)
    assert np.all(batch.dir[batch.cls == W.BE] == -1)
    assert (batch.num_q_heads, batch.num_kv_heads) == HEADS[c]
    assert batch.head_dim == 128
    assert batch.dtype == ("f32" if c == 1 else "bf16")
    for k, (lo, hi) in RANGES[c].items():
        sel = batch.ctx_lens[batch.cls == k]
        assert sel.min() >= lo and sel.max() <= hi


def test_tables_in_range_and_padded(batch):
    nblk = (batch.ctx_lens + 15) // 16
    assert batch.max_blocks_per_seq == nblk.max()
    for s in range(batch.num_seqs):
        row = batch.block_tables[s]
        assert np.all(row[:nblk[s]] >= 0) and np.all(row[:nblk[s]] < batch.num_blocks)
        assert np.all(row[nblk[s]:] == -1)


def test_no_slot_owned_twice_and_occupancy(batch):
    counts = oracle.slot_owner_counts(batch.block_tables, batch.dir, batch.ctx_lens, batch.num_blocks)
    assert counts.max() <= 1
    used_blocks = (counts.sum(axis=1) > 0).sum()
    c = batch.meta["config"]
    if c == 4:
        assert 0.895 <= used_blocks / batch.num_blocks <= 0.9
    if c == 5:
        assert used_blocks == batch.num_blocks     # pool 100 % occupied
    if c in (2, 3):
        assert batch.num_blocks == 40000
    if c == 1:
        assert batch.num_blocks == 64


def test_bidirectional_sharing_present(batch):
    if batch.meta["config"] == 1:
        return  # four sequences may or may not have fitting tails
    assert batch.meta["shared_tail_pairs"] > 0
    # a shared block appears in exactly one RT row and one BE row
    flat = {}
    for s in range(batch.num_seqs):
        n = (batch.ctx_lens[s] + 15) // 16
        for b in batch.block_tables[s, :n]:
            flat.setdefault(int(b), []).append(s)
    shared = [v for v in flat.values() if len(v) > 1]
    assert len(shared) == batch.meta["shared_tail_pairs"]
    for owners in shared:
        assert sorted(batch.cls[owners].tolist()) == [W.RT, W.BE]


def test_step_structure(batch):
    c = batch.meta["config"]
    S = batch.num_seqs
    new = np.diff(batch.cu_new)
    if c == 3:
        assert batch.num_prefill == 4 and np.all(batch.cls[:4] == W.RT)
        assert np.all(new[:4] == 512) and np.all(new[4:] == 1)
        assert np.all(batch.pos0[:4] >= 0) and np.all(batch.pos0[:4] <= 2048)
        assert batch.q_prefill.shape == (2048, 32, 128)
        assert batch.q_decode.shape == (128, 32, 128)
    else:
        assert batch.num_prefill == 0 and np.all(new == 1)
        assert batch.q_decode.shape == (S, batch.num_q_heads, 128)
    assert np.array_equal(batch.pos0, batch.ctx_lens - new)
    assert batch.k_new.shape == (batch.cu_new[-1], batch.num_kv_heads, 128)


def test_pressure_lengths_and_interleaving():
    b = W.generate(5, with_pool=False)
    ctx = b.ctx_lens.astype(np.float64)
    assert 450 < ctx.mean() < 750 and 300 < ctx.std() < 700
    # some RT block id lies strictly inside the id range of a BE sequence's blocks
    rt_ids = set()
    for s in np.flatnonzero(b.cls == W.RT):
        n = (b.ctx_lens[s] + 15) // 16
        rt_ids.update(b.block_tables[s, :n].tolist())
    inside = 0
    for s in np.flatnonzero(b.cls == W.BE):
        n = (b.ctx_lens[s] + 15) // 16
        ids = b.block_tables[s, :n]
        if n >= 3:
            lo, hi = ids[:-1].min(), ids[:-1].max()
            inside += sum(1 for r in rt_ids if lo < r < hi)
    assert inside > 0


def test_seeded_determinism():
    a = W.generate(1)
    b = W.generate(1)
    for f in ("block_tables", "ctx_lens", "dir", "k_pool", "v_pool", "q_decode", "k_new"):
        assert np.array_equal(getattr(a, f), getattr(b, f))
    c = W.generate(1, seed=7)
    assert not np.array_equal(a.k_pool, c.k_pool)


def test_pool_chunks_are_independent_streams():
    full = W.pool_values(3, 5, 1100, 2, 8, "bf16")
    again = W.pool_values(3, 5, 1100, 2, 8, "bf16", threads=1)
    assert np.array_equal(full, again)


def test_custom_batch_is_consistent():
    b = W.custom([5, 11, 40, 1], [W.RT, W.BE, W.RT, W.BE], 8, 2, head_dim=16, spare_blocks=3)
    counts = oracle.slot_owner_counts(b.block_tables, b.dir, b.ctx_lens, b.num_blocks)
    assert counts.max() <= 1
    assert b.meta["shared_tail_pairs"] >= 1


def test_compact_pool_keeps_every_sequence_cache():
    # A pool cut down to the referenced blocks, through the rewritten tables,
    # holds each sequence's cache unchanged (the oracle's own gather reads it).
    b = W.custom([40, 17, 70, 9, 33], [W.RT, W.BE, W.BE, W.RT, W.RT], 8, 4, seed=21, spare_blocks=11)
    rows = [1, 2, 4]
    tab, kp, vp = W.compact_pool(b.block_tables[rows], b.ctx_lens[rows], b.k_pool, b.v_pool)
    assert kp.shape[0] < b.num_blocks
    for i, s in enumerate(rows):
        ctx = int(b.ctx_lens[s])
        full = oracle.gather_kv(b.k_pool, b.block_tables, b.dir, s, ctx)
        small = oracle.gather_kv(kp, tab, b.dir[rows], i, ctx)
        assert np.array_equal(full, small)
        assert np.array_equal(oracle.gather_kv(b.v_pool, b.block_tables, b.dir, s, ctx),
                              oracle.gather_kv(vp, tab, b.dir[rows], i, ctx))
    nb = (b.ctx_lens[rows] + 15) // 16
    assert np.all(tab[np.arange(tab.shape[1])[None, :] >= nb[:, None]] == -1)


def test_oracle_rows_runner_matches_one_oracle_call():
    # The child runner used by the full-size GPU tests gives the same float64
    # rows as a single oracle call over the whole pool.
    from tests.oracle_rows import decode_all_rows
    b = W.custom([300, 17, 1000, 64, 5, 129], [W.BE, W.RT, W.BE, W.RT, W.BE, W.RT], 16, 4, seed=22,
                 spare_blocks=5)
    ref = oracle.decode(b.q_decode, b.k_pool, b.v_pool, b.block_tables, b.dir, b.ctx_lens, b.dtype)
    assert np.array_equal(decode_all_rows(b, workers=2), ref)
