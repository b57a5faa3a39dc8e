"""Shared pieces of the GPU parity tests: tolerances, comparison against the
oracle, NaN poisoning of unowned slots, and the oracle's version of one step."""

from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle

# Parity bar: bf16 inputs max-abs 2e-2 and mean-abs 2e-3; fp32 inputs max-abs 1e-5.
BF16_MAX_ABS = 2e-2
BF16_MEAN_ABS = 2e-3
F32_MAX_ABS = 1e-5

NAN_BITS = {"bf16": np.uint16(0x7FC0), "f32": np.float32(np.nan)}


def require_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2504_09590_amd import bros  # noqa: F401  (fails loudly when the library is missing)
    return torch


def announce(msg: str) -> None:
    """Name the case before a GPU step, flushed, so a crash log says what ran."""
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


def compare(got_bits: np.ndarray, ref: np.ndarray, dtype: str, what: str = ""):
    got = oracle.widen(got_bits, dtype)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    err = np.abs(got - ref)
    mx, mean = float(err.max(initial=0.0)), float(err.mean()) if err.size else 0.0
    if dtype == "bf16":
        assert mx <= BF16_MAX_ABS and mean <= BF16_MEAN_ABS, f"{what}: max {mx:.3g} mean {mean:.3g}"
    else:
        assert mx <= F32_MAX_ABS, f"{what}: max {mx:.3g}"
    return mx, mean


def owned_mask(batch, seqs=None) -> np.ndarray:
    """[num_blocks][16] True where some sequence's valid position lives."""
    sl = slice(None) if seqs is None else seqs
    counts = oracle.slot_owner_counts(batch.block_tables[sl], batch.dir[sl], batch.ctx_lens[sl], batch.num_blocks)
    assert counts.max(initial=0) <= 1
    return counts > 0


def poison_unowned(batch, include_new_slots: bool = False):
    """Overwrite every slot no sequence owns with NaN, in both pools (in place).
    Slots that this step's kv_write fills count as owned."""
    mask = owned_mask(batch)
    blocks, slots = np.nonzero(~mask)
    for pool in (batch.k_pool, batch.v_pool):
        pool[blocks, :, slots, :] = NAN_BITS[batch.dtype]
    return batch


def oracle_step(batch, decode_seqs=None, prefill_seqs=None):
    """The oracle's step: write the new tokens, then prefill and decode on the
    written pool. Returns (k_pool, v_pool, prefill_out, decode_out)."""
    P = batch.num_prefill
    k1, v1 = oracle.kv_write(batch.k_pool, batch.v_pool, batch.k_new, batch.v_new, batch.block_tables,
                             batch.dir, batch.pos0, batch.cu_new)
    pre = None
    if P:
        pre = oracle.prefill_chunk(batch.q_prefill, batch.cu_q, k1, v1, batch.block_tables[:P], batch.dir[:P],
                                   batch.ctx_lens[:P], batch.dtype, seqs=prefill_seqs)
    dec = oracle.decode(batch.q_decode, k1, v1, batch.block_tables[P:], batch.dir[P:], batch.ctx_lens[P:],
                        batch.dtype, seqs=decode_seqs)
    return k1, v1, pre, dec


def with_direction_table(batch, frac: float = 0.5, seed: int = 0):
    """A copy of the batch whose `dir` is the paper's direction table (one flag
    per block-table entry, Sec. 6): the per-sequence flags broadcast over the
    row, then a random `frac` of the entries whose block the sequence fills
    completely flipped. A full block has no peer, so the flipped batch stays
    consistent; its slots are simply walked the other way."""
    import dataclasses
    rng = np.random.default_rng(seed)
    maxb = batch.block_tables.shape[1]
    tab = np.repeat(np.asarray(batch.dir, dtype=np.int8)[:, None], maxb, axis=1)
    for s in range(batch.num_seqs):
        full = int(batch.ctx_lens[s]) // 16
        flip = np.nonzero(rng.random(full) < frac)[0]
        tab[s, flip] = -tab[s, flip]
    return dataclasses.replace(batch, dir=np.ascontiguousarray(tab))
