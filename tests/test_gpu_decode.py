"""bros_attn_decode against the oracle, element by element.

Covers the fp32 tiny workload (bar 1e-5), the Llama-3-8B decode workload in
full (bf16 bar), NaN-poisoned unowned slots, ragged tails (ctx % 16 in
{0, 1, 15}), one token, no context, long multi-split contexts, RT sequences
walking from the right, every supported group size, direction derived from
the class, and bitwise repeatability."""

import numpy as np
import pytest

import oracle
from paper_2504_09590_amd import workload as W
from tests.gpu_helpers import announce, compare, poison_unowned, require_gpu

pytestmark = pytest.mark.gpu


def run_decode(batch, use_dir=True, repeat=1):
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    dev = bros.to_device(batch)
    P = batch.num_prefill
    out = torch.empty_like(dev.q_decode)
    max_ctx = int(batch.ctx_lens[P:].max()) if batch.num_seqs > P else 0
    code = bros.BROS_F32 if batch.dtype == "f32" else bros.BROS_BF16
    wsb = bros.bros_attn_workspace_size(0, code, batch.num_seqs - P, batch.num_q_heads, batch.head_dim, max_ctx)
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda") if wsb else None
    if ws is not None:
        ws.fill_(255)   # NaN in every float slot: nothing may read a partial the call did not write
    outs = []
    for _ in range(repeat):
        out.fill_(float("nan"))
        bros.bros_attn_decode(out, dev.q_decode, dev.k_pool, dev.v_pool, dev.block_tables[P:],
                              dev.dir[P:] if use_dir else None, dev.cls[P:], dev.ctx_lens[P:], max_ctx,
                              workspace=ws)
        torch.cuda.synchronize()
        outs.append(bros.to_host_bits(out))
    return outs if repeat > 1 else outs[0]


def ref_decode(batch, seqs=None):
    P = batch.num_prefill
    return oracle.decode(batch.q_decode, batch.k_pool, batch.v_pool, batch.block_tables[P:], batch.dir[P:],
                         batch.ctx_lens[P:], batch.dtype, seqs=seqs)


def test_tiny_f32_decode():
    b = W.generate(1)
    announce(f"decode tiny-f32 seed={b.seed} S={b.num_seqs} ctx={b.ctx_lens.tolist()}")
    compare(run_decode(b), ref_decode(b), "f32", "tiny-f32")


def test_tiny_f32_decode_poisoned():
    b = poison_unowned(W.generate(1))
    announce("decode tiny-f32 with NaN in every unowned slot")
    compare(run_decode(b), ref_decode(b), "f32", "tiny-f32 poisoned")


def test_llama3_8b_decode_full():
    b = W.generate(2)
    announce(f"decode llama3-8b S={b.num_seqs} sum_ctx={int(b.ctx_lens.sum())}")
    mx, mean = compare(run_decode(b), ref_decode(b), "bf16", "llama3-8b")
    print(f"llama3-8b decode max {mx:.3g} mean {mean:.3g}")


EDGE_CTX = [1, 2, 15, 16, 17, 31, 32, 33, 255, 511, 512, 513, 1000, 4097, 20000]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("group", [1, 2, 4, 8])
def test_edge_lengths_and_groups(dtype, group):
    hkv = 2
    ctx = EDGE_CTX if dtype == "bf16" else EDGE_CTX[:12]
    cls = [W.RT if i % 2 == 0 else W.BE for i in range(len(ctx))]
    b = W.custom(ctx, cls, num_q_heads=hkv * group, num_kv_heads=hkv, dtype=dtype, seed=100 + group,
                 spare_blocks=7)
    poison_unowned(b)
    announce(f"decode edges dtype={dtype} G={group} ctx={ctx}")
    compare(run_decode(b), ref_decode(b), dtype, f"edges {dtype} G={group}")


def test_rt_walking_from_the_right_and_be_from_the_left():
    ctx = [5, 40, 17, 70, 16, 3]
    cls = [W.RT, W.RT, W.BE, W.BE, W.RT, W.BE]
    dirs = [-1, -1, 1, 1, 1, -1]
    b = W.custom(ctx, cls, 32, 8, dirs=dirs, share_tails=False, seed=7, spare_blocks=3)
    poison_unowned(b)
    announce("decode explicit directions against class defaults")
    compare(run_decode(b), ref_decode(b), "bf16", "explicit dirs")


def test_direction_from_class_when_flags_are_null():
    b = poison_unowned(W.custom([33, 18, 70, 9], [W.RT, W.BE, W.BE, W.RT], 32, 8, seed=8))
    announce("decode dir=NULL (from class)")
    assert np.array_equal(run_decode(b, use_dir=False), run_decode(b, use_dir=True))
    compare(run_decode(b, use_dir=False), ref_decode(b), "bf16", "dir from class")


def test_zero_context_gives_zero_row():
    b = W.custom([40, 1, 20], [W.RT, W.BE, W.RT], 8, 8, seed=9)
    b.ctx_lens[1] = 0
    announce("decode with a zero-length context")
    got = run_decode(b)
    ref = ref_decode(b)
    assert np.all(oracle.widen(got[1], "bf16") == 0)
    compare(got, ref, "bf16", "zero ctx")


def test_repeatable_bitwise():
    b = W.custom([3000, 77, 9000, 16], [W.BE, W.RT, W.BE, W.RT], 32, 8, seed=10)
    announce("decode twice, bitwise")
    a, c = run_decode(b, repeat=2)
    assert np.array_equal(a, c)


def test_shared_tail_blocks_are_read_per_sequence():
    # Every RT tail shares its block with a BE tail; poison the rest.
    ctx = [16 * 3 + 5, 16 * 2 + 11, 7, 9, 16 * 10 + 1, 15]
    cls = [W.RT, W.BE, W.RT, W.BE, W.RT, W.BE]
    b = W.custom(ctx, cls, 32, 8, seed=11)
    assert b.meta["shared_tail_pairs"] >= 2
    poison_unowned(b)
    announce("decode over shared RT/BE tail blocks")
    compare(run_decode(b), ref_decode(b), "bf16", "shared tails")


def _oracle_rows_in_child(config, out_path):
    """Start the oracle over every decode row of workload `config` in a child
    process (it regenerates the workload from its seed and never touches the
    GPU); returns the process."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    return subprocess.Popen([sys.executable, "-m", "tests.oracle_rows", str(config), str(out_path)], cwd=root)


@pytest.mark.parametrize("config", [4, 5])
def test_full_size_workloads_every_row(config, tmp_path):
    # The 70B-shaped (G = 8, ctx up to 16384) and memory-pressure (512 rows,
    # 100 % occupied pool, RT blocks inside BE runs) workloads in the launch
    # the benchmark times; every row is compared with the oracle, which runs
    # in a child process meanwhile.
    ref_path = tmp_path / f"oracle_{config}.npy"
    child = _oracle_rows_in_child(config, ref_path)
    try:
        b = W.generate(config)
        announce(f"decode {b.name} S={b.num_seqs} sum_ctx={int(b.ctx_lens.sum())} (every row)")
        got = run_decode(b)
    finally:
        rc = child.wait(timeout=600)
    assert rc == 0, f"oracle child exited with {rc}"
    ref = np.load(ref_path)
    mx, mean = compare(got, ref, "bf16", f"{b.name} every row")
    print(f"{b.name} decode, all {ref.shape[0]} rows: max {mx:.3g} mean {mean:.3g}")


def test_more_rows_than_the_prefix_holds_in_lds():
    # Above 4096 rows the per-row tile prefix is kept per chunk of rows.
    rng = np.random.default_rng(12)
    n = 4500
    ctx = rng.integers(1, 49, n)
    cls = [W.RT if i % 3 == 0 else W.BE for i in range(n)]
    b = W.custom(ctx, cls, 8, 8, seed=12, spare_blocks=9)
    poison_unowned(b)
    announce(f"decode {n} rows, ctx 1..48")
    compare(run_decode(b), ref_decode(b), "bf16", "4500 rows")


def test_workspace_reused_across_batches():
    # Partials left in a workspace by one call must not leak into the next.
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    a = W.custom([9000, 40, 3000, 17], [W.BE, W.RT, W.BE, W.RT], 32, 8, seed=13)
    c = W.custom([5000, 2000, 33, 700, 12000], [W.BE, W.BE, W.RT, W.RT, W.BE], 32, 8, seed=14)
    wsb = max(bros.bros_attn_workspace_size(0, bros.BROS_BF16, x.num_seqs, 32, 128, int(x.ctx_lens.max()))
              for x in (a, c))
    ws = torch.full((wsb,), 0x7F, dtype=torch.uint8, device="cuda")   # finite garbage everywhere
    announce("decode two batches through one workspace")
    outs = []
    for x in (a, c, a):
        dev = bros.to_device(x)
        out = torch.empty_like(dev.q_decode)
        bros.bros_attn_decode(out, dev.q_decode, dev.k_pool, dev.v_pool, dev.block_tables, dev.dir, dev.cls,
                              dev.ctx_lens, int(x.ctx_lens.max()), workspace=ws)
        torch.cuda.synchronize()
        outs.append(bros.to_host_bits(out))
    compare(outs[0], ref_decode(a), "bf16", "first batch")
    compare(outs[1], ref_decode(c), "bf16", "second batch")
    assert np.array_equal(outs[0], outs[2])


def test_calls_on_two_streams_at_once():
    # Calls on different streams with workspaces of their own may run at the
    # same time: the library keeps no state between calls but per-device
    # queries, so each gives what it gives alone.
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    a = W.custom([9000, 40, 3000, 17, 700], [W.BE, W.RT, W.BE, W.RT, W.BE], 32, 8, seed=15)
    c = W.custom([5000, 2000, 33, 12000], [W.BE, W.BE, W.RT, W.BE], 32, 8, seed=16)
    devs, outs, wss = [], [], []
    for x in (a, c):
        dev = bros.to_device(x)
        devs.append(dev)
        outs.append(torch.full_like(dev.q_decode, float("nan")))
        wsb = bros.bros_attn_workspace_size(0, bros.BROS_BF16, x.num_seqs, 32, 128, int(x.ctx_lens.max()))
        wss.append(torch.full((wsb,), 255, dtype=torch.uint8, device="cuda"))
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    announce("decode on two streams at once")
    for _ in range(3):
        for x, dev, out, ws, st in zip((a, c), devs, outs, wss, streams):
            bros.bros_attn_decode(out, dev.q_decode, dev.k_pool, dev.v_pool, dev.block_tables, dev.dir, dev.cls,
                                  dev.ctx_lens, int(x.ctx_lens.max()), workspace=ws, stream=st)
    torch.cuda.synchronize()
    compare(bros.to_host_bits(outs[0]), ref_decode(a), "bf16", "stream 1")
    compare(bros.to_host_bits(outs[1]), ref_decode(c), "bf16", "stream 2")
