"""bros_attn_mixed: the prefill chunks and the decode rows of one batch in one
launch (the concatenated batch of Sec. 6), against the oracle's step and
against the two separate calls; with few prefill units (workgroups without a
unit take only decode work), every group size, NaN-poisoned unowned slots, a
per-entry direction table, rows without context, and the dispatch cases (one
half only, more prefill units than one grid holds)."""

import numpy as np
import pytest

from paper_2504_09590_amd import workload as W
from tests.gpu_helpers import announce, compare, oracle_step, poison_unowned, require_gpu, with_direction_table

pytestmark = pytest.mark.gpu


def _run(batch, fused):
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    from paper_2504_09590_amd.step import MixedStep
    dev = bros.to_device(batch)
    step = MixedStep(batch, dev, fused=fused)
    for ws in (step.ws_decode, step.ws_prefill):
        if ws is not None:
            ws.fill_(255)   # NaN in every float slot: nothing may read a partial the call did not write
    step.out_prefill.fill_(float("nan"))
    step.out_decode.fill_(float("nan"))
    pre, dec = step.run()
    torch.cuda.synchronize()
    return (bros.to_host_bits(dev.k_pool), bros.to_host_bits(dev.v_pool), bros.to_host_bits(pre),
            bros.to_host_bits(dec))


def _check(batch, what):
    k_ref, v_ref, pre_ref, dec_ref = oracle_step(batch)
    k, v, pre, dec = _run(batch, fused=True)
    assert np.array_equal(k, k_ref) and np.array_equal(v, v_ref), f"{what}: pools after the write"
    if batch.num_prefill:
        compare(pre, pre_ref, batch.dtype, f"{what} prefill")
    if batch.num_seqs > batch.num_prefill:
        compare(dec, dec_ref, batch.dtype, f"{what} decode")
    return pre, dec


def test_fused_mixed_step_workload():
    b = W.generate(3)
    announce(f"fused mixed step {b.name} seed={b.seed}")
    pre, dec = _check(b, "fused mixed step")
    # the prefill units run the same code as the prefill call: identical rows
    _, _, pre2, dec2 = _run(W.generate(3), fused=False)
    assert np.array_equal(pre, pre2)
    compare(dec, __import__("oracle").widen(dec2, "bf16"), "bf16", "fused vs separate decode")


@pytest.mark.parametrize("group", [1, 2, 4, 8])
def test_fused_small_batches_every_group(group):
    hkv = 2
    # two prefill chunks (one on cached context), decode rows with short,
    # ragged, long and zero contexts
    ctx = [300 + 40, 77, 1, 16, 17, 4097, 900, 33]
    cls = [W.RT, W.RT, W.BE, W.RT, W.BE, W.BE, W.RT, W.BE]
    new = [40, 77, 1, 1, 1, 1, 1, 1]
    b = W.custom(ctx, cls, hkv * group, hkv, seed=50 + group, num_prefill=2, new_counts=new, spare_blocks=5)
    poison_unowned(b)
    announce(f"fused small batch G={group}")
    _check(b, f"fused G={group}")


def test_fused_direction_table_and_empty_rows():
    ctx = [64 + 130, 45, 2000, 0, 700, 31]
    cls = [W.RT, W.RT, W.BE, W.BE, W.RT, W.BE]
    new = [130, 45, 1, 0, 1, 1]
    b = W.custom(ctx, cls, 32, 8, seed=61, num_prefill=2, new_counts=new, spare_blocks=3)
    b = with_direction_table(b, frac=0.5, seed=61)
    poison_unowned(b)
    announce("fused with a per-entry direction table and a decode row without context")
    _, dec = _check(b, "fused direction table")
    import oracle
    assert np.all(oracle.widen(dec[3 - 2], "bf16") == 0)


def test_fused_dispatch_one_half_and_too_many_units():
    # decode rows only, prefill chunks only, and 8 chunks of 512 rows (1024
    # prefill units: more than one grid, so the two calls run in turn)
    only_dec = W.custom([500, 37, 1200], [W.BE, W.RT, W.BE], 32, 8, seed=71)
    announce("fused dispatch: decode only")
    _check(only_dec, "decode only")
    only_pre = W.custom([100, 600], [W.RT, W.RT], 32, 8, seed=72, num_prefill=2, new_counts=[100, 512])
    announce("fused dispatch: prefill only")
    _check(only_pre, "prefill only")
    ctx = [512 + 50 * i for i in range(8)] + [3000, 700]
    many = W.custom(ctx, [W.RT] * 8 + [W.BE, W.BE], 32, 8, seed=73, num_prefill=8,
                    new_counts=[512] * 8 + [1, 1])
    announce("fused dispatch: 1024 prefill units")
    _check(many, "two calls in turn")


def test_fused_pool_rows_past_32_bit_offsets():
    """More than 2^20 (block, KV head) rows: the fused grid's prefill units take
    the 64-bit address path; the batch's blocks sit past 4 GiB of each pool."""
    torch = require_gpu()
    import oracle
    from paper_2504_09590_amd import bros
    b = W.custom([300 + 200, 77, 900, 33], [W.RT, W.RT, W.BE, W.BE], 32, 8, seed=81, num_prefill=2,
                 new_counts=[200, 77, 1, 1], spare_blocks=3)
    announce("fused, pool rows past 2^20")
    k_ref, v_ref, pre_ref, dec_ref = oracle_step(b)
    # the oracle's pools after the write: the kernels read them, no write here
    b.k_pool, b.v_pool = k_ref, v_ref
    shift = (1 << 17) + 3
    dev = bros.to_device(b)
    big_k = torch.empty((shift + b.num_blocks,) + tuple(dev.k_pool.shape[1:]), dtype=dev.k_pool.dtype, device="cuda")
    big_v = torch.empty_like(big_k)
    big_k[shift:] = dev.k_pool
    big_v[shift:] = dev.v_pool
    tables = dev.block_tables.clone()
    tables[tables >= 0] += shift
    P = b.num_prefill
    hq = b.num_q_heads
    out_p = torch.full_like(dev.q_prefill, float("nan"))
    out_d = torch.full_like(dev.q_decode, float("nan"))
    max_pre = int(b.ctx_lens[:P].max())
    max_dec = int(b.ctx_lens[P:].max())
    wsb = bros.bros_attn_workspace_size(bros.BROS_WS_DECODE, bros.BROS_BF16, b.num_seqs - P, hq, b.head_dim, max_dec)
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
    bros.bros_attn_mixed(out_p, dev.q_prefill, dev.cu_q, int(np.diff(b.cu_q).max()), max_pre, out_d, dev.q_decode,
                         max_dec, big_k, big_v, tables, dev.dir, dev.cls, dev.ctx_lens, P, workspace=ws)
    torch.cuda.synchronize()
    compare(bros.to_host_bits(out_p), pre_ref, "bf16", "fused prefill, pool rows past 2^20")
    compare(bros.to_host_bits(out_d), dec_ref, "bf16", "fused decode, pool rows past 2^20")
    del big_k, big_v
    torch.cuda.empty_cache()
