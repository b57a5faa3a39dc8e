"""Seeded synthetic batches for the mixed RT/BE paged-attention step.

This module only draws inputs: sequence lengths, classes, direction flags, block
tables that emulate the bidirectional block manager's output (Sec. 5.2: a BE
request's last block may be shared with an RT request's last block, the RT
tokens filling it from the left and the BE tokens from the right, so an RT tail
of r tokens and a BE tail of b tokens share one block when r + b <= 16), and
N(0, 1) tensor values. It holds no attention arithmetic and no slot mapping; the
HIP path and the oracle both consume what it returns.

The paper measures on ShareGPT / LMSYS-Chat traces and a synthetic BE set; none
of those are used here. Every batch below is synthetic, with the shapes, length
ranges and pool occupancies of five named workloads:

  tiny-f32-decode        4 sequences (2 RT, 2 BE), 8 q = 8 KV heads, fp32,
                         ctx U{17..300}, 64-block pool, random permutation tables
  llama3-8b-decode       64 sequences (16 RT ctx U{128..2048}, 48 BE ctx
                         U{1024..8192}), 32 q / 8 KV heads, bf16, 40000-block pool
  llama3-8b-mixed-step   4 RT prefill chunks of 512 new tokens on top of
                         c0 U{0..2048} cached tokens, then 128 BE decode
                         sequences (ctx U{512..8192}), bf16, 40000-block pool
  llama3-70b-decode      288 sequences (32 RT ctx U{256..4096}, 256 BE ctx
                         U{2048..16384}), 64 q / 8 KV heads, bf16, pool sized
                         for 90 % occupancy with the free blocks scattered
  llama3-8b-pressure     512 sequences (25 % RT), ctx log-normal with mean 600
                         and sd 500 clipped to [16, 32768], bf16, pool 100 %
                         occupied, RT blocks interleaved inside BE block runs

Integer "U{a..b}" is inclusive on both ends. bf16 values are fp32 N(0, 1) draws
rounded to nearest-even. Tensors are numpy arrays; bf16 tensors are uint16 bit
patterns.
"""

from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

BLOCK_SIZE = 16
RT, BE = 0, 1
DIR_OF_CLASS = {RT: 1, BE: -1}   # RT fills from the left, BE from the right

# Values are drawn in chunks of this many blocks, each from its own seeded
# stream, so that any subset of the pool can be regenerated independently.
_CHUNK_BLOCKS = 512


@dataclass
class Batch:
    name: str
    dtype: str                      # "f32" or "bf16"
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    num_blocks: int
    block_tables: np.ndarray        # int32 [S][max_blocks]; -1 beyond each sequence's blocks
    dir: np.ndarray                 # int8 [S], +1 or -1
    cls: np.ndarray                 # uint8 [S], 0 = RT, 1 = BE
    ctx_lens: np.ndarray            # int32 [S], tokens cached after this step's writes
    num_prefill: int                # sequences [0, num_prefill) are prefill chunks
    cu_q: np.ndarray                # int32 [num_prefill + 1], prefill query rows
    q_prefill: np.ndarray           # [Tq][Hq][D]
    q_decode: np.ndarray            # [S - num_prefill][Hq][D]
    cu_new: np.ndarray              # int32 [S + 1], new tokens per sequence
    pos0: np.ndarray                # int32 [S], position of each sequence's first new token
    k_new: np.ndarray               # [Tn][Hkv][D]
    v_new: np.ndarray
    k_pool: np.ndarray              # [num_blocks][Hkv][16][D]
    v_pool: np.ndarray
    seed: int
    meta: dict = field(default_factory=dict)

    @property
    def num_seqs(self) -> int:
        return int(self.ctx_lens.shape[0])

    @property
    def max_blocks_per_seq(self) -> int:
        return int(self.block_tables.shape[1])

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def max_ctx(self) -> int:
        return int(self.ctx_lens.max()) if self.num_seqs else 0

    def decode_slice(self):
        """Metadata rows of the decode sequences (they follow the prefill ones)."""
        p = self.num_prefill
        return slice(p, self.num_seqs)


# ---------------------------------------------------------------------------
# values
# ---------------------------------------------------------------------------

def _to_bf16_bits(x32: np.ndarray) -> np.ndarray:
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def _normal(seed: int, tag: int, shape, dtype: str) -> np.ndarray:
    rng = np.random.default_rng([seed, tag])
    x = rng.standard_normal(shape, dtype=np.float32)
    return x if dtype == "f32" else _to_bf16_bits(x)


def pool_values(seed: int, tag: int, num_blocks: int, hkv: int, d: int, dtype: str,
                threads: int = 8) -> np.ndarray:
    """[num_blocks][Hkv][16][D] N(0, 1) values; chunk c of _CHUNK_BLOCKS blocks
    comes from stream (seed, tag, c)."""
    np_dtype = np.float32 if dtype == "f32" else np.uint16
    out = np.empty((num_blocks, hkv, BLOCK_SIZE, d), dtype=np_dtype)
    n_chunks = (num_blocks + _CHUNK_BLOCKS - 1) // _CHUNK_BLOCKS

    def fill(c):
        lo = c * _CHUNK_BLOCKS
        hi = min(num_blocks, lo + _CHUNK_BLOCKS)
        rng = np.random.default_rng([seed, tag, c])
        x = rng.standard_normal((hi - lo, hkv, BLOCK_SIZE, d), dtype=np.float32)
        out[lo:hi] = x if dtype == "f32" else _to_bf16_bits(x)

    if n_chunks <= 1 or threads <= 1:
        for c in range(n_chunks):
            fill(c)
    else:
        with ThreadPoolExecutor(max_workers=threads) as ex:
            list(ex.map(fill, range(n_chunks)))
    return out


# ---------------------------------------------------------------------------
# block allocation (emulates the block manager's output)
# ---------------------------------------------------------------------------

def _tails(ctx: np.ndarray) -> np.ndarray:
    """Tokens in each sequence's last block (1..16)."""
    return ctx - BLOCK_SIZE * ((ctx + BLOCK_SIZE - 1) // BLOCK_SIZE - 1)


def pair_tails(ctx: np.ndarray, cls: np.ndarray):
    """Greedy RT/BE last-block sharing: each RT sequence, in order, takes the
    unpaired BE sequence with the largest tail b that still fits (r + b <= 16).
    Returns {rt_index: be_index}."""
    tails = _tails(ctx)
    free = {b: [] for b in range(1, BLOCK_SIZE + 1)}
    for i in np.flatnonzero(cls == BE):
        free[int(tails[i])].append(int(i))
    for b in free:
        free[b].reverse()            # pop() then yields the lowest index first
    pairs = {}
    for i in np.flatnonzero(cls == RT):
        r = int(tails[i])
        for b in range(BLOCK_SIZE - r, 0, -1):
            if free[b]:
                pairs[int(i)] = free[b].pop()
                break
    return pairs


def _block_counts(ctx):
    return ((ctx + BLOCK_SIZE - 1) // BLOCK_SIZE).astype(np.int64)


def _tables_from_ids(ctx, pairs, ids_iter_fn):
    """Assign physical ids to every (sequence, block index); a paired RT
    sequence's last block reuses its BE partner's last block id."""
    nblk = _block_counts(ctx)
    S = len(ctx)
    maxb = int(nblk.max()) if S else 1
    tables = np.full((S, maxb), -1, dtype=np.int32)
    for s in range(S):
        n = int(nblk[s])
        own = n - 1 if s in pairs else n
        tables[s, :own] = ids_iter_fn(s, own)
    for rt, be in pairs.items():
        tables[rt, nblk[rt] - 1] = tables[be, nblk[be] - 1]
    return tables


def _needed_blocks(ctx, pairs) -> int:
    return int(_block_counts(ctx).sum()) - len(pairs)


def allocate_permuted(rng, ctx, cls, num_blocks):
    """Block ids drawn in order from a random permutation of the pool."""
    pairs = pair_tails(ctx, cls)
    need = _needed_blocks(ctx, pairs)
    if need > num_blocks:
        return None
    perm = rng.permutation(num_blocks).astype(np.int32)
    cursor = [0]

    def take(s, n):
        ids = perm[cursor[0]:cursor[0] + n]
        cursor[0] += n
        return ids

    return _tables_from_ids(ctx, pairs, take), pairs


def allocate_interleaved_full(rng, ctx, cls):
    """Pool 100 % occupied: BE sequences get contiguous runs of ids in shuffled
    order; RT blocks (those not sharing a BE tail) are dropped at random
    positions inside that run sequence, so they sit between BE blocks."""
    pairs = pair_tails(ctx, cls)
    nblk = _block_counts(ctx)
    own = nblk.copy()
    for rt in pairs:
        own[rt] -= 1
    be_order = rng.permutation(np.flatnonzero(cls == BE))
    rt_idx = np.flatnonzero(cls == RT)
    n_be = int(own[be_order].sum())
    n_rt = int(own[rt_idx].sum())
    total = n_be + n_rt
    rt_slots = np.zeros(total, dtype=bool)
    rt_slots[rng.choice(total, size=n_rt, replace=False)] = True
    rt_positions = np.flatnonzero(rt_slots).astype(np.int32)
    be_positions = np.flatnonzero(~rt_slots).astype(np.int32)
    start = {}
    c = 0
    for s in be_order:
        start[int(s)] = ("be", c)
        c += int(own[s])
    c = 0
    for s in rng.permutation(rt_idx):
        start[int(s)] = ("rt", c)
        c += int(own[s])

    def take(s, n):
        kind, off = start[s]
        src = be_positions if kind == "be" else rt_positions
        return src[off:off + n]

    return _tables_from_ids(ctx, pairs, take), pairs, total


# ---------------------------------------------------------------------------
# the five workloads
# ---------------------------------------------------------------------------

CONFIGS = {
    1: "tiny-f32-decode",
    2: "llama3-8b-decode",
    3: "llama3-8b-mixed-step",
    4: "llama3-70b-decode",
    5: "llama3-8b-pressure",
}
NAME_TO_CONFIG = {v: k for k, v in CONFIGS.items()}


def _shuffle_batch(rng, ctx, cls):
    order = rng.permutation(len(ctx))
    return ctx[order], cls[order]


def _lognormal_params(mean, sd):
    sigma2 = math.log(1.0 + (sd / mean) ** 2)
    return math.log(mean) - sigma2 / 2.0, math.sqrt(sigma2)


def _lengths(config: int, rng):
    """ctx lengths and classes, in batch order."""
    if config == 1:
        cls = np.array([RT, RT, BE, BE], dtype=np.uint8)
        ctx = rng.integers(17, 301, size=4)
        return _shuffle_batch(rng, ctx, cls)
    if config == 2:
        ctx = np.concatenate([rng.integers(128, 2049, 16), rng.integers(1024, 8193, 48)])
        cls = np.array([RT] * 16 + [BE] * 48, dtype=np.uint8)
        return _shuffle_batch(rng, ctx, cls)
    if config == 3:
        c0 = rng.integers(0, 2049, 4)
        ctx = np.concatenate([c0 + 512, rng.integers(512, 8193, 128)])
        cls = np.array([RT] * 4 + [BE] * 128, dtype=np.uint8)
        return ctx, cls                 # prefill chunks first, then decode
    if config == 4:
        ctx = np.concatenate([rng.integers(256, 4097, 32), rng.integers(2048, 16385, 256)])
        cls = np.array([RT] * 32 + [BE] * 256, dtype=np.uint8)
        return _shuffle_batch(rng, ctx, cls)
    if config == 5:
        mu, sigma = _lognormal_params(600.0, 500.0)
        ctx = np.clip(np.rint(rng.lognormal(mu, sigma, 512)), 16, 32768).astype(np.int64)
        cls = np.array([RT] * 128 + [BE] * 384, dtype=np.uint8)
        return _shuffle_batch(rng, ctx, cls)
    raise ValueError(f"unknown config {config}")


_SHAPES = {  # (Hq, Hkv, D, dtype)
    1: (8, 8, 128, "f32"),
    2: (32, 8, 128, "bf16"),
    3: (32, 8, 128, "bf16"),
    4: (64, 8, 128, "bf16"),
    5: (32, 8, 128, "bf16"),
}


def generate(config, seed: int | None = None, with_pool: bool = True) -> Batch:
    """Build workload `config` (1..5 or its name). Seed defaults to 1000 + config."""
    if isinstance(config, str):
        config = NAME_TO_CONFIG[config]
    seed = 1000 + config if seed is None else seed
    rng = np.random.default_rng(seed)
    hq, hkv, d, dtype = _SHAPES[config]

    for _attempt in range(1000):
        ctx, cls = _lengths(config, rng)
        ctx = ctx.astype(np.int64)
        if config in (1, 2, 3):
            num_blocks = {1: 64, 2: 40000, 3: 40000}[config]
            got = allocate_permuted(rng, ctx, cls, num_blocks)
            if got is None:
                continue           # redraw lengths with the next values of the stream
            tables, pairs = got
        elif config == 4:
            pairs = pair_tails(ctx, cls)
            num_blocks = int(math.ceil(_needed_blocks(ctx, pairs) / 0.9))
            tables, pairs = allocate_permuted(rng, ctx, cls, num_blocks)
        else:
            tables, pairs, num_blocks = allocate_interleaved_full(rng, ctx, cls)
        break
    else:
        raise RuntimeError("could not draw a batch that fits the pool")

    S = len(ctx)
    dirs = np.array([DIR_OF_CLASS[int(c)] for c in cls], dtype=np.int8)
    num_prefill = 4 if config == 3 else 0
    new_counts = np.ones(S, dtype=np.int64)
    if num_prefill:
        new_counts[:num_prefill] = 512
    cu_new = np.concatenate([[0], np.cumsum(new_counts)]).astype(np.int32)
    pos0 = (ctx - new_counts).astype(np.int32)
    cu_q = np.concatenate([[0], np.cumsum(new_counts[:num_prefill])]).astype(np.int32)

    tn = int(cu_new[-1])
    q_prefill = _normal(seed, 1, (int(cu_q[-1]), hq, d), dtype)
    q_decode = _normal(seed, 2, (S - num_prefill, hq, d), dtype)
    k_new = _normal(seed, 3, (tn, hkv, d), dtype)
    v_new = _normal(seed, 4, (tn, hkv, d), dtype)
    if with_pool:
        k_pool = pool_values(seed, 5, num_blocks, hkv, d, dtype)
        v_pool = pool_values(seed, 6, num_blocks, hkv, d, dtype)
    else:
        k_pool = v_pool = np.empty((0, hkv, BLOCK_SIZE, d), dtype=np.float32 if dtype == "f32" else np.uint16)

    return Batch(
        name=CONFIGS[config], dtype=dtype, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
        num_blocks=int(num_blocks), block_tables=tables, dir=dirs, cls=cls.astype(np.uint8),
        ctx_lens=ctx.astype(np.int32), num_prefill=num_prefill, cu_q=cu_q,
        q_prefill=q_prefill, q_decode=q_decode, cu_new=cu_new, pos0=pos0,
        k_new=k_new, v_new=v_new, k_pool=k_pool, v_pool=v_pool, seed=seed,
        meta={"config": config, "shared_tail_pairs": len(pairs)},
    )


def custom(ctx, cls, num_q_heads, num_kv_heads, head_dim=128, dtype="bf16", seed=0,
           num_prefill=0, new_counts=None, spare_blocks=0, dirs=None, share_tails=True) -> Batch:
    """A small batch with caller-chosen lengths and classes (for edge cases).

    Sequences [0, num_prefill) get new_counts[s] new rows each (a prefill chunk);
    the rest get one new token. Tables come from a random permutation of a pool
    with `spare_blocks` unowned blocks; RT/BE tails share blocks when
    share_tails is set. `dirs` overrides the class-derived direction flags."""
    rng = np.random.default_rng(seed)
    ctx = np.asarray(ctx, dtype=np.int64)
    cls = np.asarray(cls, dtype=np.uint8)
    S = len(ctx)
    pairs = pair_tails(ctx, cls) if share_tails else {}
    num_blocks = max(1, _needed_blocks(ctx, pairs) + spare_blocks)
    perm = rng.permutation(num_blocks).astype(np.int32)
    cursor = [0]

    def take(s, n):
        ids = perm[cursor[0]:cursor[0] + n]
        cursor[0] += n
        return ids

    tables = _tables_from_ids(ctx, pairs, take) if S else np.full((0, 1), -1, np.int32)
    if dirs is None:
        dirs = np.array([DIR_OF_CLASS[int(c)] for c in cls], dtype=np.int8)
    else:
        dirs = np.asarray(dirs, dtype=np.int8)
    if new_counts is None:
        new_counts = np.ones(S, dtype=np.int64)
    new_counts = np.asarray(new_counts, dtype=np.int64)
    cu_new = np.concatenate([[0], np.cumsum(new_counts)]).astype(np.int32)
    pos0 = (ctx - new_counts).astype(np.int32)
    cu_q = np.concatenate([[0], np.cumsum(new_counts[:num_prefill])]).astype(np.int32)
    hq, hkv, d = num_q_heads, num_kv_heads, head_dim
    tn = int(cu_new[-1])
    return Batch(
        name="custom", dtype=dtype, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
        num_blocks=int(num_blocks), block_tables=tables, dir=dirs, cls=cls,
        ctx_lens=ctx.astype(np.int32), num_prefill=num_prefill, cu_q=cu_q,
        q_prefill=_normal(seed, 1, (int(cu_q[-1]), hq, d), dtype),
        q_decode=_normal(seed, 2, (S - num_prefill, hq, d), dtype),
        cu_new=cu_new, pos0=pos0,
        k_new=_normal(seed, 3, (tn, hkv, d), dtype), v_new=_normal(seed, 4, (tn, hkv, d), dtype),
        k_pool=pool_values(seed, 5, int(num_blocks), hkv, d, dtype),
        v_pool=pool_values(seed, 6, int(num_blocks), hkv, d, dtype),
        seed=seed, meta={"shared_tail_pairs": len(pairs)},
    )


# ---------------------------------------------------------------------------
# a pool holding only the blocks some sequences reference
# ---------------------------------------------------------------------------

def compact_pool(block_tables, ctx_lens, k_pool, v_pool):
    """The pool blocks that entries [0, ceil(ctx / 16)) of these table rows
    reference, renumbered 0 .. n-1 in id order, and the rows rewritten to the
    new ids (-1 in every other entry). A sequence's cache is the same through
    the new rows and the smaller pool, so a consumer that reads only the blocks
    a table references sees the same values with far less memory. Entries
    outside [0, num_blocks) stay -1."""
    tables = np.asarray(block_tables)
    ctx = np.asarray(ctx_lens, dtype=np.int64)
    nblk = _block_counts(np.maximum(ctx, 0))
    used = np.arange(tables.shape[1])[None, :] < nblk[:, None]
    ids = tables[used]
    ids = np.unique(ids[(ids >= 0) & (ids < k_pool.shape[0])])
    remap = np.full(k_pool.shape[0], -1, dtype=np.int64)
    remap[ids] = np.arange(len(ids))
    ok = used & (tables >= 0) & (tables < k_pool.shape[0])
    out = np.full(tables.shape, -1, dtype=np.int32)
    out[ok] = remap[tables[ok]]
    return out, k_pool[ids], v_pool[ids]
