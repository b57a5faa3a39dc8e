"""bros_kv_write is bit-exact: every written slot holds the source bytes and
every other byte of both pools is unchanged (the random initial pool acts as a
canary everywhere). Includes RT and BE tails sharing one block, written in the
same launch."""

import numpy as np
import pytest

import oracle
from paper_2504_09590_amd import workload as W
from tests.gpu_helpers import announce, require_gpu

pytestmark = pytest.mark.gpu


def run_write(batch):
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    dev = bros.to_device(batch)
    bros.bros_kv_write(dev.k_new, dev.v_new, dev.k_pool, dev.v_pool, dev.block_tables, dev.dir, dev.cls,
                       dev.pos0, dev.cu_new)
    torch.cuda.synchronize()
    return dev


def check_bitwise(batch, dev):
    from paper_2504_09590_amd import bros
    k1, v1 = oracle.kv_write(batch.k_pool, batch.v_pool, batch.k_new, batch.v_new, batch.block_tables,
                             batch.dir, batch.pos0, batch.cu_new)
    for name, ref, got in (("k", k1, dev.k_pool), ("v", v1, dev.v_pool)):
        g = bros.to_host_bits(got)
        assert g.dtype == ref.dtype
        same = g.view(np.uint8) == np.ascontiguousarray(ref).view(np.uint8)
        assert same.all(), f"{name}_pool differs at {np.count_nonzero(~same)} bytes"


@pytest.mark.parametrize("config", [1, 3])
def test_workload_writes(config):
    b = W.generate(config)
    announce(f"kv_write {b.name} tokens={int(b.cu_new[-1])}")
    check_bitwise(b, run_write(b))


def test_shared_tails_written_in_one_launch():
    # each RT tail shares a block with a BE tail; both write their next token now
    ctx = [16 + 6, 16 * 3 + 10, 5, 11, 16 * 4 + 16, 1]
    cls = [W.RT, W.BE, W.RT, W.BE, W.RT, W.BE]
    b = W.custom(ctx, cls, 8, 8, seed=40)
    assert b.meta["shared_tail_pairs"] >= 2
    announce("kv_write shared tails")
    check_bitwise(b, run_write(b))


@pytest.mark.parametrize("num_seqs,num_prefill", [(600, 0), (300, 3)])
def test_more_sequences_than_threads(num_seqs, num_prefill):
    # a workgroup's 256 threads each check one sequence's range per pass:
    # sequences 256 and up are found on the later passes
    rng = np.random.default_rng(43 + num_seqs)
    ctx = [int(x) for x in rng.integers(1, 90, num_seqs)]
    cls = [W.RT if i % 3 == 0 else W.BE for i in range(num_seqs)]
    new_counts = None
    if num_prefill:
        new_counts = [1] * num_seqs
        for s in range(num_prefill):
            ctx[s] = 40 + 37 * s
            new_counts[s] = 20 + 7 * s
    b = W.custom(ctx, cls, 8, 8, seed=44 + num_seqs, num_prefill=num_prefill, new_counts=new_counts)
    announce(f"kv_write {num_seqs} sequences, {num_prefill} chunks, tokens={int(b.cu_new[-1])}")
    check_bitwise(b, run_write(b))


def test_prefill_chunks_and_fp32():
    b = W.custom([300, 40, 7, 90], [W.RT, W.RT, W.BE, W.BE], 8, 2, dtype="f32", seed=41, num_prefill=2,
                 new_counts=[130, 40, 1, 1], spare_blocks=4)
    announce("kv_write fp32 with 130- and 40-token chunks")
    check_bitwise(b, run_write(b))


@pytest.mark.parametrize("hkv,dtype", [(1, "bf16"), (3, "bf16"), (5, "f32"), (24, "bf16"), (40, "f32")])
def test_kv_head_counts(hkv, dtype):
    # a token's chunks are split into (token, tensor, head, chunk) by a quotient
    # with a runtime divisor (chunks per token); head counts that are not powers
    # of two, and counts whose chunks take several passes of the workgroup
    b = W.custom([37, 16, 5, 70, 2], [W.RT, W.BE, W.BE, W.RT, W.RT], hkv, hkv, dtype=dtype, seed=50 + hkv,
                 num_prefill=1, new_counts=[21, 1, 1, 1, 1], spare_blocks=3)
    announce(f"kv_write Hkv={hkv} {dtype}")
    check_bitwise(b, run_write(b))


def test_direction_from_class_when_flags_are_null():
    # dir = NULL: each sequence's direction comes from its class (RT from the
    # left end, BE from the right end), as the flags would give it
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    b = W.custom([16 + 6, 16 * 3 + 10, 5, 11, 70], [W.RT, W.BE, W.RT, W.BE, W.BE], 8, 8, seed=42,
                 num_prefill=1, new_counts=[22, 1, 1, 1, 1])
    assert np.array_equal(b.dir, np.where(b.cls == W.RT, 1, -1).astype(np.int8))
    dev = bros.to_device(b)
    announce("kv_write with null direction flags")
    bros.bros_kv_write(dev.k_new, dev.v_new, dev.k_pool, dev.v_pool, dev.block_tables, None, dev.cls,
                       dev.pos0, dev.cu_new)
    torch.cuda.synchronize()
    check_bitwise(b, dev)
