"""bros_attn_prefill_chunk against the oracle.

The pools are written by the oracle's kv_write first (so the chunk's own K/V
are in place) and then uploaded, so these tests exercise the prefill kernel
alone. Covers the mixed-step workload's four 512-row chunks (with the
workspace and without), a long-context chunk whose units are split over their
keys when they leave compute units idle, an empty chunk between others, the
longest context of the matrix-core path (its whole table in LDS; split into
128 pieces per unit with the workspace), more units than the device-side plan
holds, c0 = 0 (pure causal), chunk starts and lengths off the 16/64 grid, one-row chunks, RT
chunks walking from the right, all group sizes, the fp32 path, NaN-poisoned
unowned slots, the last row against a decode at the same length, and a pool
whose rows lie past 32-bit byte offsets."""

import numpy as np
import pytest

import oracle
from paper_2504_09590_amd import workload as W
from tests.gpu_helpers import announce, compare, poison_unowned, require_gpu

pytestmark = pytest.mark.gpu


def written(batch):
    """The batch with the oracle's kv_write applied to its pools."""
    k1, v1 = oracle.kv_write(batch.k_pool, batch.v_pool, batch.k_new, batch.v_new, batch.block_tables,
                             batch.dir, batch.pos0, batch.cu_new)
    batch.k_pool, batch.v_pool = k1, v1
    return batch


def run_prefill(batch, workspace=True, ws_bytes=None, stream=None):
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    dev = bros.to_device(batch)
    P = batch.num_prefill
    out = torch.full_like(dev.q_prefill, float("nan"))
    max_ctx = int(batch.ctx_lens[:P].max())
    max_q = int(np.diff(batch.cu_q).max())
    code = bros.BROS_F32 if batch.dtype == "f32" else bros.BROS_BF16
    wsb = bros.bros_attn_workspace_size(1, code, int(batch.cu_q[-1]), batch.num_q_heads, batch.head_dim, max_ctx)
    if ws_bytes is not None:
        wsb = ws_bytes
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda") if wsb and workspace else None
    if ws is not None:
        ws.fill_(255)   # NaN in every float slot: nothing may read a partial the call did not write
    bros.bros_attn_prefill_chunk(out, dev.q_prefill, dev.cu_q, max_q, dev.k_pool, dev.v_pool,
                                 dev.block_tables[:P], dev.dir[:P], dev.cls[:P], dev.ctx_lens[:P], max_ctx,
                                 workspace=ws, stream=stream)
    torch.cuda.synchronize()
    return bros.to_host_bits(out)


def ref_prefill(batch):
    P = batch.num_prefill
    return oracle.prefill_chunk(batch.q_prefill, batch.cu_q, batch.k_pool, batch.v_pool, batch.block_tables[:P],
                                batch.dir[:P], batch.ctx_lens[:P], batch.dtype)


def chunk_batch(c0s, ns, classes, group=4, hkv=8, dtype="bf16", seed=0, dirs=None, extra_decode=()):
    """Prefill sequences first (ctx = c0 + n), then optional decode sequences."""
    ctx = [c + n for c, n in zip(c0s, ns)] + list(extra_decode)
    cls = list(classes) + [W.BE] * len(extra_decode)
    new = list(ns) + [1] * len(extra_decode)
    if dirs is not None:
        dirs = list(dirs) + [-1] * len(extra_decode)
    return W.custom(ctx, cls, hkv * group, hkv, dtype=dtype, seed=seed, num_prefill=len(ns), new_counts=new,
                    spare_blocks=5, dirs=dirs)


@pytest.mark.parametrize("workspace", [True, False], ids=["workspace", "no-workspace"])
def test_mixed_step_workload_prefill_chunks(workspace):
    b = written(W.generate(3))
    announce(f"prefill llama3-8b-mixed-step chunks c0={(b.ctx_lens[:4] - 512).tolist()} workspace={workspace}")
    mx, mean = compare(run_prefill(b, workspace), ref_prefill(b), "bf16", "mixed-step prefill")
    print(f"prefill max {mx:.3g} mean {mean:.3g}")


@pytest.mark.parametrize("group,hkv", [(4, 2), (1, 8)])
def test_long_context_chunk_split_into_pieces(group, hkv):
    # fewer (row tile, KV head) units than compute units, one of them over ~390
    # key tiles: with the workspace the long units are cut into pieces over
    # their keys and merged. Both forms match the oracle; they differ from each
    # other by rounding, which shows the split path ran.
    b = written(chunk_batch([12000, 0, 7], [512, 64, 1], [W.RT] * 3, group=group, hkv=hkv, seed=34 + group))
    poison_unowned(b)
    announce(f"prefill c0=12000 n=512 beside short chunks G={group} Hkv={hkv} (split pieces)")
    split, whole = run_prefill(b), run_prefill(b, workspace=False)
    ref = ref_prefill(b)
    compare(split, ref, "bf16", "long-context split")
    compare(whole, ref, "bf16", "long-context whole units")
    assert not np.array_equal(split, whole)
    # a workspace smaller than the query is accepted and splits nothing
    assert np.array_equal(run_prefill(b, ws_bytes=4096), whole)


def test_split_on_a_compute_unit_share():
    # the split sizes its pieces by the stream's compute units: 96 units on a
    # 128-CU share are still split (and 128 more ranks launched)
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    b = written(chunk_batch([12000, 0, 7], [512, 64, 1], [W.RT] * 3, group=4, hkv=2, seed=38))
    poison_unowned(b)
    announce("prefill split on a 128-CU stream")
    share = bros.bros_stream_create_cu_share(0, 128)
    try:
        got = run_prefill(b, stream=share)
    finally:
        torch.cuda.synchronize()
        bros.bros_stream_destroy(share)
    compare(got, ref_prefill(b), "bf16", "split on a CU share")


def test_empty_chunk_between_others():
    # a sequence with no new rows in the length table is skipped; its neighbours are not
    b = written(chunk_batch([10, 50, 0], [40, 0, 65], [W.RT] * 3, group=4, hkv=2, seed=36))
    poison_unowned(b)
    announce("prefill with an empty chunk between two others")
    compare(run_prefill(b), ref_prefill(b), "bf16", "empty chunk")


@pytest.mark.parametrize("workspace", [False, True], ids=["whole", "split"])
def test_longest_context_of_the_matrix_core_path(workspace):
    # ctx = 32768 exactly: the whole 2048-entry table staged in LDS; with the
    # workspace the two units (one KV head) are cut into 128 pieces each
    b = written(chunk_batch([32768 - 40], [40], [W.RT], group=4, hkv=1, seed=37))
    assert int(b.ctx_lens[0]) == 32768
    poison_unowned(b)
    announce(f"prefill ctx 32768 (the matrix-core path's limit), workspace={workspace}")
    compare(run_prefill(b, workspace), ref_prefill(b), "bf16", f"ctx 32768 {'split' if workspace else 'whole'}")


def test_more_units_than_the_device_plan_holds():
    # 17 chunks of 512 rows at G=4: 272 units per KV head, past the 256 the
    # kernels plan on the device; every unit runs whole
    c0 = [int(x) for x in np.random.default_rng(35).integers(0, 300, 17)]
    b = written(chunk_batch(c0, [512] * 17, [W.RT] * 17, group=4, hkv=2, seed=35))
    announce("prefill 17 x 512-row chunks (unit fallback)")
    compare(run_prefill(b), ref_prefill(b), "bf16", "272 units")


@pytest.mark.parametrize("group", [1, 2, 4, 8])
def test_ragged_chunks_all_groups(group):
    b = written(chunk_batch([0, 5, 16, 1000, 63], [37, 1, 100, 300, 65], [W.RT] * 5, group=group, hkv=2,
                            seed=20 + group, extra_decode=(9, 40)))
    poison_unowned(b)
    announce(f"prefill ragged chunks G={group}")
    compare(run_prefill(b), ref_prefill(b), "bf16", f"ragged G={group}")


def test_pure_causal_and_single_row():
    b = written(chunk_batch([0, 0, 77], [128, 1, 1], [W.RT, W.RT, W.RT], seed=30))
    poison_unowned(b)
    announce("prefill c0=0 and one-row chunks")
    compare(run_prefill(b), ref_prefill(b), "bf16", "causal/single")


def test_rt_chunks_walking_from_the_right():
    b = written(chunk_batch([19, 200], [45, 70], [W.RT, W.RT], dirs=[-1, 1], seed=31))
    poison_unowned(b)
    announce("prefill with a right-to-left RT chunk")
    compare(run_prefill(b), ref_prefill(b), "bf16", "dir -1 chunk")


def test_f32_chunks():
    b = written(chunk_batch([0, 21, 300], [20, 33, 17], [W.RT] * 3, group=4, hkv=2, dtype="f32", seed=32))
    poison_unowned(b)
    announce("prefill fp32 (vector path)")
    compare(run_prefill(b), ref_prefill(b), "f32", "f32 prefill")


def test_last_row_matches_decode_at_the_same_length():
    b = written(chunk_batch([90], [40], [W.RT], seed=33))
    got = oracle.widen(run_prefill(b), "bf16")[-1]
    ref = oracle.decode(b.q_prefill[-1:], b.k_pool, b.v_pool, b.block_tables[:1], b.dir[:1], b.ctx_lens[:1], "bf16")[0]
    assert np.abs(got - ref).max() <= 2e-2


def test_bf16_context_beyond_the_matrix_core_path():
    # max_ctx above 32768 routes bf16 prefill through the decode kernel in row
    # mode (every chunk row a decode row with its own causal context).
    b = written(chunk_batch([33000], [40], [W.RT], group=4, hkv=1, seed=15))
    poison_unowned(b)
    announce("prefill bf16 c0=33000 n=40 (row-mode path)")
    compare(run_prefill(b), ref_prefill(b), "bf16", "bf16 ctx > 32768")


def test_pool_rows_past_32_bit_offsets():
    """A pool of more than 2^20 (block, KV head) rows: the loads take the
    64-bit address path. The batch's blocks sit past the first 4 GiB of each
    pool (the rows below are left unwritten and never read)."""
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    b = written(chunk_batch([300, 40, 0], [200, 130, 77], [W.RT, W.BE, W.RT], group=4, hkv=8, seed=77))
    announce("prefill, pool rows past 2^20")
    ref = ref_prefill(b)
    shift = (1 << 17) + 5            # x 8 KV heads x 4 KiB: past 4 GiB
    dev = bros.to_device(b)
    big_k = torch.empty((shift + b.num_blocks,) + tuple(dev.k_pool.shape[1:]), dtype=dev.k_pool.dtype, device="cuda")
    big_v = torch.empty_like(big_k)
    big_k[shift:] = dev.k_pool
    big_v[shift:] = dev.v_pool
    tables = dev.block_tables.clone()
    tables[tables >= 0] += shift
    P = b.num_prefill
    out = torch.full_like(dev.q_prefill, float("nan"))
    max_ctx = int(b.ctx_lens[:P].max())
    bros.bros_attn_prefill_chunk(out, dev.q_prefill, dev.cu_q, int(np.diff(b.cu_q).max()), big_k, big_v,
                                 tables[:P], dev.dir[:P], dev.cls[:P], dev.ctx_lens[:P], max_ctx)
    torch.cuda.synchronize()
    compare(bros.to_host_bits(out), ref, "bf16", "prefill, pool rows past 2^20")
    del big_k, big_v
    torch.cuda.empty_cache()
