"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these checks re-types the oracle's own formulas: the layout is pinned by
a hand-enumerated fixture of Sec. 5.1/5.2, the attention arithmetic by torch's
scaled_dot_product_attention (an independent library routine) and by brute
force on tiny inputs, and the rest by invariants that a dropped term, a wrong
sign or index, or a transposed operand would break. The last test plants such
mistakes in the oracle and checks that some pin catches each one.
"""

import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import paged_attention as pa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLDEN = os.path.join(ROOT, "tests", "golden", "bidirectional_layout.json")
GOLDEN_PER_ENTRY = os.path.join(ROOT, "tests", "golden", "per_entry_direction.json")


def _load_golden():
    with open(GOLDEN) as f:
        return json.load(f)


def _golden_batch(hkv=2, d=8, seed=0):
    g = _load_golden()
    S = len(g["sequences"])
    maxb = max(len(s["block_table"]) for s in g["sequences"])
    tables = np.zeros((S, maxb), dtype=np.int32)
    dirs = np.zeros(S, dtype=np.int8)
    ctx = np.zeros(S, dtype=np.int32)
    for i, s in enumerate(g["sequences"]):
        tables[i, :len(s["block_table"])] = s["block_table"]
        dirs[i] = s["dir"]
        ctx[i] = s["ctx"]
    rng = np.random.default_rng(seed)
    shape = (g["num_blocks"], hkv, g["block_size"], d)
    k_pool = rng.standard_normal(shape).astype(np.float32)
    v_pool = rng.standard_normal(shape).astype(np.float32)
    return g, tables, dirs, ctx, k_pool, v_pool


def _per_entry_batch(hkv=2, d=8, seed=0):
    """The per-entry fixture as arrays: tables and the [S][max_blocks] flag
    table, with pool values drawn from a seeded normal."""
    with open(GOLDEN_PER_ENTRY) as f:
        g = json.load(f)
    seqs = g["sequences"]
    tables = np.array([s["block_table"] for s in seqs], dtype=np.int32)
    flags = np.array([s["dir_per_entry"] for s in seqs], dtype=np.int8)
    ctx = np.array([s["ctx"] for s in seqs], dtype=np.int32)
    rng = np.random.default_rng(seed)
    shape = (g["num_blocks"], hkv, g["block_size"], d)
    k_pool = rng.standard_normal(shape).astype(np.float32)
    v_pool = rng.standard_normal(shape).astype(np.float32)
    return g, tables, flags, ctx, k_pool, v_pool


def _contiguous_batch(rng, ctxs, hkv, d, poison=True):
    """Pool built by a plain reshape of each sequence's contiguous K/V (direction
    +1, consecutive blocks); unused tail slots hold NaN."""
    nblk = [(c + 15) // 16 for c in ctxs]
    nb = sum(nblk)
    k_pool = np.full((nb, hkv, 16, d), np.nan if poison else 0.0, dtype=np.float32)
    v_pool = k_pool.copy()
    tables = np.zeros((len(ctxs), max(nblk)), dtype=np.int32)
    dense_k, dense_v = [], []
    off = 0
    for s, c in enumerate(ctxs):
        K = rng.standard_normal((c, hkv, d)).astype(np.float32)
        V = rng.standard_normal((c, hkv, d)).astype(np.float32)
        dense_k.append(K)
        dense_v.append(V)
        for name, dense, pool in (("k", K, k_pool), ("v", V, v_pool)):
            padded = np.full((nblk[s] * 16, hkv, d), np.nan, dtype=np.float32)
            padded[:c] = dense
            pool[off:off + nblk[s]] = padded.reshape(nblk[s], 16, hkv, d).transpose(0, 2, 1, 3)
        tables[s, :nblk[s]] = np.arange(off, off + nblk[s])
        off += nblk[s]
    dirs = np.ones(len(ctxs), dtype=np.int8)
    return k_pool, v_pool, tables, dirs, dense_k, dense_v


def _sdpa(q, K, V, mask=None, causal=False):
    """torch SDPA in float64: q [n, Hq, D], K/V [ctx, Hkv, D] -> [n, Hq, D]."""
    qt = torch.from_numpy(np.ascontiguousarray(q, dtype=np.float64)).permute(1, 0, 2)[None]
    kt = torch.from_numpy(np.ascontiguousarray(K, dtype=np.float64)).permute(1, 0, 2)[None]
    vt = torch.from_numpy(np.ascontiguousarray(V, dtype=np.float64)).permute(1, 0, 2)[None]
    am = None if mask is None else torch.from_numpy(mask)
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=am,
                                                         is_causal=causal, enable_gqa=True)
    return o[0].permute(1, 0, 2).numpy()


# ----------------------------------------------------------------------------
# pins, written as functions so the mutation test can re-run them
# ----------------------------------------------------------------------------

def pin_golden_positions():
    g, tables, dirs, ctx, _, _ = _golden_batch()
    for s, seq in enumerate(g["sequences"]):
        blocks, slots = oracle.physical_location(tables, dirs, s, np.arange(seq["ctx"]))
        got = [[int(b), int(sl)] for b, sl in zip(blocks, slots)]
        assert got == seq["position_to_block_slot"], seq["name"]


def pin_golden_uniform_query():
    """q = 0 gives equal weights, so the output is the plain mean of exactly the
    V rows the fixture lists; a wrong slot or a leaked slot changes it."""
    g, tables, dirs, ctx, k_pool, v_pool = _golden_batch()
    hq = 4
    q = np.zeros((len(ctx), hq, k_pool.shape[-1]), dtype=np.float32)
    out = oracle.decode(q, k_pool, v_pool, tables, dirs, ctx, "f32")
    group = hq // k_pool.shape[1]
    for s, seq in enumerate(g["sequences"]):
        rows = np.array([v_pool[b, :, sl, :] for b, sl in seq["position_to_block_slot"]], dtype=np.float64)
        mean = rows.mean(axis=0)  # [Hkv, D]
        for h in range(hq):
            np.testing.assert_allclose(out[s, h], mean[h // group], rtol=0, atol=1e-13)


def pin_per_entry_positions():
    """Each table entry is walked in its own flag's direction."""
    g, tables, flags, ctx, _, _ = _per_entry_batch()
    for s, seq in enumerate(g["sequences"]):
        blocks, slots = oracle.physical_location(tables, flags, s, np.arange(seq["ctx"]))
        got = [[int(b), int(sl)] for b, sl in zip(blocks, slots)]
        assert got == seq["position_to_block_slot"], seq["name"]


def pin_per_entry_attention_vs_sdpa():
    """Decode and a prefill chunk over the per-entry fixture equal dense SDPA
    over the K/V rows the fixture lists, in its order (the rows of the other
    slots are NaN, so a leaked slot shows)."""
    g, tables, flags, ctx, k_pool, v_pool = _per_entry_batch(hkv=2, d=8, seed=3)
    owned = {(b, sl) for seq in g["sequences"] for b, sl in seq["position_to_block_slot"]}
    for b in range(k_pool.shape[0]):
        for sl in range(16):
            if (b, sl) not in owned:
                k_pool[b, :, sl, :] = np.nan
                v_pool[b, :, sl, :] = np.nan
    rng = np.random.default_rng(4)
    hq = 4
    q = rng.standard_normal((len(ctx), hq, 8)).astype(np.float32)
    out = oracle.decode(q, k_pool, v_pool, tables, flags, ctx, "f32")
    dense = []
    for s, seq in enumerate(g["sequences"]):
        K = np.array([k_pool[b, :, sl, :] for b, sl in seq["position_to_block_slot"]])
        V = np.array([v_pool[b, :, sl, :] for b, sl in seq["position_to_block_slot"]])
        dense.append((K, V))
        np.testing.assert_allclose(out[s], _sdpa(q[s:s + 1], K, V)[0], rtol=0, atol=1e-12)
    # the last 9 positions of X as a chunk on its first 31
    n = 9
    qp = rng.standard_normal((n, hq, 8)).astype(np.float32)
    got = oracle.prefill_chunk(qp, np.array([0, n], dtype=np.int32), k_pool, v_pool, tables[:1], flags[:1],
                               ctx[:1], "f32")
    K, V = dense[0]
    c0 = int(ctx[0]) - n
    mask = np.arange(int(ctx[0]))[None, :] <= (c0 + np.arange(n))[:, None]
    np.testing.assert_allclose(got, _sdpa(qp, K, V, mask=mask), rtol=0, atol=1e-12)


def pin_sdpa_decode():
    rng = np.random.default_rng(11)
    ctxs = [1, 15, 16, 17, 40, 123]
    hq, hkv, d = 8, 2, 16
    k_pool, v_pool, tables, dirs, dk, dv = _contiguous_batch(rng, ctxs, hkv, d)
    q = rng.standard_normal((len(ctxs), hq, d)).astype(np.float32)
    out = oracle.decode(q, k_pool, v_pool, tables, dirs, np.array(ctxs), "f32")
    for s in range(len(ctxs)):
        ref = _sdpa(q[s:s + 1], dk[s], dv[s])
        np.testing.assert_allclose(out[s], ref[0], rtol=0, atol=1e-12)


def pin_sdpa_prefill():
    rng = np.random.default_rng(12)
    ctxs = [37, 64, 90]
    news = [37, 20, 1]          # c0 = 0 (pure causal), 44, 89
    hq, hkv, d = 4, 4, 8
    k_pool, v_pool, tables, dirs, dk, dv = _contiguous_batch(rng, ctxs, hkv, d)
    cu_q = np.concatenate([[0], np.cumsum(news)]).astype(np.int32)
    q = rng.standard_normal((cu_q[-1], hq, d)).astype(np.float32)
    out = oracle.prefill_chunk(q, cu_q, k_pool, v_pool, tables, dirs, np.array(ctxs), "f32")
    for s in range(len(ctxs)):
        rows = slice(cu_q[s], cu_q[s + 1])
        c0 = ctxs[s] - news[s]
        if c0 == 0:
            ref = _sdpa(q[rows], dk[s], dv[s], causal=True)
        else:
            qpos = c0 + np.arange(news[s])
            mask = np.arange(ctxs[s])[None, :] <= qpos[:, None]
            ref = _sdpa(q[rows], dk[s], dv[s], mask=mask)
        np.testing.assert_allclose(out[rows], ref, rtol=0, atol=1e-12)


def pin_bruteforce_tiny():
    """S=1, one head, D=2, three tokens, scale 1: weights 1, e, e^2 by hand."""
    k_pool = np.zeros((1, 1, 16, 2), dtype=np.float32)
    v_pool = np.zeros((1, 1, 16, 2), dtype=np.float32)
    # BE direction: positions 0, 1, 2 sit in slots 15, 14, 13 (right end first).
    k_pool[0, 0, 15] = [0.0, 5.0]
    k_pool[0, 0, 14] = [1.0, -3.0]
    k_pool[0, 0, 13] = [2.0, 7.0]
    v_pool[0, 0, 15] = [1.0, 0.0]
    v_pool[0, 0, 14] = [0.0, 1.0]
    v_pool[0, 0, 13] = [1.0, 1.0]
    k_pool[0, 0, :13] = np.nan
    v_pool[0, 0, :13] = np.nan
    q = np.array([[[1.0, 0.0]]], dtype=np.float32)
    out = oracle.decode(q, k_pool, v_pool, np.array([[0]]), np.array([-1]), np.array([3]), "f32", scale=1.0)
    e = math.e
    total = 1 + e + e * e
    expect = [(1 + e * e) / total, (e + e * e) / total]
    np.testing.assert_allclose(out[0, 0], expect, rtol=0, atol=1e-15)


def pin_gqa_vs_sdpa_grouping():
    """With grouped heads the convention is torch's enable_gqa one: head h reads
    KV head h // (Hq // Hkv)."""
    rng = np.random.default_rng(13)
    ctxs = [29, 50]
    hq, hkv, d = 8, 2, 8
    k_pool, v_pool, tables, dirs, dk, dv = _contiguous_batch(rng, ctxs, hkv, d)
    q = rng.standard_normal((2, hq, d)).astype(np.float32)
    out = oracle.decode(q, k_pool, v_pool, tables, dirs, np.array(ctxs), "f32")
    for s in range(2):
        rep_k = np.repeat(dk[s], hq // hkv, axis=1)
        rep_v = np.repeat(dv[s], hq // hkv, axis=1)
        ref = _sdpa(q[s:s + 1], rep_k, rep_v)
        np.testing.assert_allclose(out[s], ref[0], rtol=0, atol=1e-12)


ALL_PINS = [pin_golden_positions, pin_golden_uniform_query, pin_per_entry_positions,
            pin_per_entry_attention_vs_sdpa, pin_sdpa_decode, pin_sdpa_prefill, pin_bruteforce_tiny,
            pin_gqa_vs_sdpa_grouping]


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin()


# ----------------------------------------------------------------------------
# invariants on random bidirectional batches
# ----------------------------------------------------------------------------

def _random_shared_batch(rng, n_pairs=3, n_solo=2, hkv=2, d=16, dtype="f32"):
    """RT/BE pairs whose tails share one block (r + b <= 16), plus unshared
    sequences. Built by hand-rolled allocation, independent of any generator."""
    ctxs, dirs = [], []
    for _ in range(n_pairs):
        r = int(rng.integers(1, 16))
        b = int(rng.integers(1, 17 - r))
        ctxs += [16 * int(rng.integers(0, 4)) + r, 16 * int(rng.integers(0, 4)) + b]
        dirs += [1, -1]
    for _ in range(n_solo):
        ctxs.append(int(rng.integers(1, 70)))
        dirs.append(int(rng.choice([1, -1])))
    nblk = [(c + 15) // 16 for c in ctxs]
    total = sum(nblk) - n_pairs
    perm = rng.permutation(total + 5)  # 5 spare blocks nobody owns
    tables = np.zeros((len(ctxs), max(nblk)), dtype=np.int32)
    nxt = 0
    for s in range(len(ctxs)):
        for i in range(nblk[s]):
            if s < 2 * n_pairs and s % 2 == 1 and i == nblk[s] - 1:
                tables[s, i] = tables[s - 1, nblk[s - 1] - 1]  # BE tail joins the RT tail's block
            else:
                tables[s, i] = perm[nxt]
                nxt += 1
    nb = total + 5
    shape = (nb, hkv, 16, d)
    k_pool = rng.standard_normal(shape).astype(np.float32)
    v_pool = rng.standard_normal(shape).astype(np.float32)
    return k_pool, v_pool, tables, np.array(dirs, dtype=np.int8), np.array(ctxs, dtype=np.int32)


def test_random_batches_are_disjoint():
    rng = np.random.default_rng(5)
    for _ in range(20):
        _, _, tables, dirs, ctx = _random_shared_batch(rng)
        oracle.owned_slots(tables, dirs, ctx)


def test_owned_slots_rejects_overlap():
    # RT tail of 9 and BE tail of 8 in one block: 9 + 8 > 16, slot 8 collides.
    tables = np.array([[0], [0]], dtype=np.int32)
    with pytest.raises(ValueError):
        oracle.owned_slots(tables, np.array([1, -1]), np.array([9, 8]))


def test_pool_permutation_is_bitwise_invariant():
    rng = np.random.default_rng(6)
    k, v, t, d, c = _random_shared_batch(rng)
    q = rng.standard_normal((len(c), 4, k.shape[-1])).astype(np.float32)
    base = oracle.decode(q, k, v, t, d, c, "f32")
    pi = rng.permutation(k.shape[0])          # new id of old block b is pi[b]
    k2 = np.empty_like(k)
    v2 = np.empty_like(v)
    k2[pi] = k
    v2[pi] = v
    got = oracle.decode(q, k2, v2, pi[t].astype(np.int32), d, c, "f32")
    assert np.array_equal(base, got)


def test_direction_flip_with_mirrored_pool_is_bitwise_invariant():
    rng = np.random.default_rng(7)
    k, v, t, d, c = _random_shared_batch(rng)
    q = rng.standard_normal((len(c), 4, k.shape[-1])).astype(np.float32)
    base = oracle.decode(q, k, v, t, d, c, "f32")
    got = oracle.decode(q, k[:, :, ::-1, :], v[:, :, ::-1, :], t, -d, c, "f32")
    assert np.array_equal(base, got)


def test_per_entry_direction_table_matches_per_sequence():
    rng = np.random.default_rng(8)
    k, v, t, d, c = _random_shared_batch(rng)
    q = rng.standard_normal((len(c), 4, k.shape[-1])).astype(np.float32)
    per_entry = np.repeat(d[:, None], t.shape[1], axis=1)
    assert np.array_equal(oracle.decode(q, k, v, t, d, c, "f32"),
                          oracle.decode(q, k, v, t, per_entry, c, "f32"))


def test_unowned_slots_never_read():
    rng = np.random.default_rng(9)
    k, v, t, d, c = _random_shared_batch(rng)
    owner = oracle.owned_slots(t, d, c)
    k2, v2 = k.copy(), v.copy()
    for b in range(k.shape[0]):
        for sl in range(16):
            if (b, sl) not in owner:
                k2[b, :, sl, :] = np.nan
                v2[b, :, sl, :] = np.inf
    q = rng.standard_normal((len(c), 4, k.shape[-1])).astype(np.float32)
    assert np.array_equal(oracle.decode(q, k, v, t, d, c, "f32"),
                          oracle.decode(q, k2, v2, t, d, c, "f32"))


def test_prefill_row_equals_decode_at_that_length():
    rng = np.random.default_rng(10)
    k, v, t, d, c = _random_shared_batch(rng, n_pairs=2, n_solo=1)
    s = int(np.argmax(c))
    n = min(int(c[s]), 9)
    q = rng.standard_normal((n, 4, k.shape[-1])).astype(np.float32)
    cu_q = np.zeros(len(c) + 1, dtype=np.int32)
    cu_q[s + 1:] = n
    pre = oracle.prefill_chunk(q, cu_q, k, v, t, d, c, "f32")
    c0 = int(c[s]) - n
    for j in range(n):
        ctx_j = c.copy()
        ctx_j[s] = c0 + j + 1
        qd = np.zeros((len(c), 4, k.shape[-1]), dtype=np.float32)
        qd[s] = q[j]
        dec = oracle.decode(qd, k, v, t, d, ctx_j, "f32", seqs=[s])
        np.testing.assert_allclose(pre[j], dec[s], rtol=0, atol=1e-14)


def test_chunked_prefill_equals_one_chunk():
    """Write 12 tokens and attend once, or write+attend 5 then 7: same rows."""
    rng = np.random.default_rng(14)
    hkv, hq, dd = 2, 4, 8
    c0, n = 19, 12
    nb = 4
    table = np.array([[3, 1, 0]], dtype=np.int32)
    for direction in (1, -1):
        dirs = np.array([direction], dtype=np.int8)
        k0 = rng.standard_normal((nb, hkv, 16, dd)).astype(np.float32)
        v0 = rng.standard_normal((nb, hkv, 16, dd)).astype(np.float32)
        kn = rng.standard_normal((n, hkv, dd)).astype(np.float32)
        vn = rng.standard_normal((n, hkv, dd)).astype(np.float32)
        q = rng.standard_normal((n, hq, dd)).astype(np.float32)
        k1, v1 = oracle.kv_write(k0, v0, kn, vn, table, dirs, [c0], [0, n])
        whole = oracle.prefill_chunk(q, [0, n], k1, v1, table, dirs, [c0 + n], "f32")
        ka, va = oracle.kv_write(k0, v0, kn[:5], vn[:5], table, dirs, [c0], [0, 5])
        part1 = oracle.prefill_chunk(q[:5], [0, 5], ka, va, table, dirs, [c0 + 5], "f32")
        kb, vb = oracle.kv_write(ka, va, kn[5:], vn[5:], table, dirs, [c0 + 5], [0, 7])
        part2 = oracle.prefill_chunk(q[5:], [0, 7], kb, vb, table, dirs, [c0 + n], "f32")
        np.testing.assert_allclose(whole, np.concatenate([part1, part2]), rtol=0, atol=1e-14)


def test_kv_write_places_golden_tokens_and_keeps_canaries():
    """Writing every position of the fixture's sequences, token by token, puts
    token p of a sequence exactly at the fixture's (block, slot) and changes no
    other byte."""
    g, tables, dirs, ctx, _, _ = _golden_batch()
    hkv, d = 2, 4
    canary = np.float32(-12345.5)
    k_pool = np.full((4, hkv, 16, d), canary, dtype=np.float32)
    v_pool = k_pool.copy()
    cu = np.concatenate([[0], np.cumsum(ctx)]).astype(np.int32)
    k_new = np.zeros((cu[-1], hkv, d), dtype=np.float32)
    v_new = np.zeros((cu[-1], hkv, d), dtype=np.float32)
    for s in range(len(ctx)):
        for p in range(ctx[s]):
            k_new[cu[s] + p] = 1000 * s + p
            v_new[cu[s] + p] = -(1000 * s + p)
    k1, v1 = oracle.kv_write(k_pool, v_pool, k_new, v_new, tables, dirs, [0, 0, 0], cu)
    seen = np.zeros((4, 16), dtype=bool)
    for s, seq in enumerate(g["sequences"]):
        for p, (b, sl) in enumerate(seq["position_to_block_slot"]):
            assert np.all(k1[b, :, sl, :] == 1000 * s + p)
            assert np.all(v1[b, :, sl, :] == -(1000 * s + p))
            seen[b, sl] = True
    assert seen.all()  # the fixture fills all four blocks


def test_kv_write_leaves_unwritten_slots_bitwise():
    rng = np.random.default_rng(15)
    k, v, t, d, c = _random_shared_batch(rng)
    new = np.ones(len(c), dtype=np.int32)
    cu = np.concatenate([[0], np.cumsum(new)]).astype(np.int32)
    kn = rng.standard_normal((cu[-1], k.shape[1], k.shape[-1])).astype(np.float32)
    vn = rng.standard_normal((cu[-1], k.shape[1], k.shape[-1])).astype(np.float32)
    pos0 = c - 1
    k1, v1 = oracle.kv_write(k, v, kn, vn, t, d, pos0, cu)
    changed = np.any(k1.view(np.uint32) != k.view(np.uint32), axis=(1, 3))
    assert changed.sum() <= len(c)
    for s in range(len(c)):
        b, sl = oracle.physical_location(t, d, s, [c[s] - 1])
        assert np.array_equal(k1[b[0], :, sl[0], :], kn[s])
        assert np.array_equal(v1[b[0], :, sl[0], :], vn[s])


def test_bf16_widening_matches_torch():
    rng = np.random.default_rng(16)
    x = torch.from_numpy(rng.standard_normal(1000).astype(np.float32)).to(torch.bfloat16)
    bits = x.view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oracle.widen(bits, "bf16"), x.to(torch.float64).numpy())


def test_decode_without_context_is_zero():
    k = np.ones((1, 1, 16, 4), dtype=np.float32)
    out = oracle.decode(np.ones((1, 1, 4), dtype=np.float32), k, k, np.array([[0]]),
                        np.array([1]), np.array([0]), "f32")
    assert np.all(out == 0)


def test_direction_flags_must_be_signed_unit():
    with pytest.raises(ValueError):
        oracle.slot_in_block(3, 0)


# ----------------------------------------------------------------------------
# planted mistakes: every one must trip at least one pin
# ----------------------------------------------------------------------------

def _mutant_ignore_direction(p, direction):
    return np.asarray(p) % 16


def _mutant_inverted_direction(p, direction):
    off = np.asarray(p) % 16
    return np.where(np.asarray(direction) == 1, 15 - off, off)


def _mutant_block_index_swapped(block_tables, dir_flags, s, positions):
    positions = np.asarray(positions, dtype=np.int64)
    bi = np.minimum(positions % 16, np.asarray(block_tables).shape[1] - 1)
    blocks = np.asarray(block_tables)[s][bi].astype(np.int64)
    return blocks, pa.slot_in_block(positions, pa._direction_of(dir_flags, s, bi))


def _mutant_gqa_modulo(q, k, v, limits, scale):
    n, hq, d = q.shape
    hkv = k.shape[1]
    out = np.zeros((n, hq, d))
    for h in range(hq):
        out[:, h:h + 1] = _ORIG_SOFTMAX(q[:, h:h + 1], k[:, h % hkv:h % hkv + 1], v[:, h % hkv:h % hkv + 1], limits, scale)
    return out


def _mutant_exclusive_diagonal(q, k, v, limits, scale):
    return _ORIG_SOFTMAX(q, k, v, np.maximum(np.asarray(limits) - 1, 1), scale)


def _mutant_transposed_pv(q, k, v, limits, scale):
    return _ORIG_SOFTMAX(q, v, k, limits, scale)


def _mutant_first_entry_direction(dir_flags, s, block_index):
    dir_flags = np.asarray(dir_flags)
    flag = dir_flags[s] if dir_flags.ndim == 1 else dir_flags[s][0]
    return np.broadcast_to(flag, np.shape(block_index))


_ORIG_SOFTMAX = pa.softmax_attention

MUTANTS = {
    "ignore_direction": ("slot_in_block", _mutant_ignore_direction),
    "inverted_direction": ("slot_in_block", _mutant_inverted_direction),
    "block_index_swapped": ("physical_location", _mutant_block_index_swapped),
    "gqa_modulo": ("softmax_attention", _mutant_gqa_modulo),
    "exclusive_causal_diagonal": ("softmax_attention", _mutant_exclusive_diagonal),
    "k_v_swapped": ("softmax_attention", _mutant_transposed_pv),
    "scale_dropped": ("default_scale", lambda d: 1.0),
    "per_entry_flags_collapsed": ("_direction_of", _mutant_first_entry_direction),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(monkeypatch, name):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(pa, attr, fn)
    caught = []
    for pin in ALL_PINS:
        try:
            pin()
        except (AssertionError, ValueError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"mutant {name} survived every pin"
