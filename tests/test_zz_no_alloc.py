"""bros_attn_decode_noalloc (the decode entry point that allocates nothing;
its workspace is the library's static scratch array) against bros_attn_decode
with a caller workspace and against the oracle: two calls in a row, the second
on a smaller batch, through the C ABI. Same kernels, so the outputs must be
bitwise equal; both must meet the bf16 parity bar against the oracle."""

import ctypes

import numpy as np
import pytest

import oracle
from paper_2504_09590_amd import workload as W
from tests.gpu_helpers import announce, compare, require_gpu

pytestmark = pytest.mark.gpu


def _noalloc_via_c_abi(bros, out, dev, max_ctx):
    """The new entry point called directly through the C ABI (ctypes)."""
    nb, hkv, bs, d = (int(x) for x in dev.k_pool.shape)
    st = bros.LIB.bros_attn_decode_noalloc(
        ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(dev.q_decode.data_ptr()),
        ctypes.c_void_p(dev.k_pool.data_ptr()), ctypes.c_void_p(dev.v_pool.data_ptr()), nb,
        ctypes.c_void_p(dev.block_tables.data_ptr()), int(dev.block_tables.shape[1]),
        ctypes.c_void_p(dev.dir.data_ptr()), ctypes.c_void_p(dev.cls.data_ptr()), 0,
        ctypes.c_void_p(dev.ctx_lens.data_ptr()), int(max_ctx), int(dev.ctx_lens.shape[0]),
        int(dev.q_decode.shape[1]), hkv, d, bs, 0.0, bros.BROS_BF16, None)
    assert st == 0, bros.LIB.bros_last_error().decode()


def _both(batch):
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    dev = bros.to_device(batch)
    max_ctx = int(batch.ctx_lens.max())
    wsb = bros.bros_attn_workspace_size(bros.BROS_WS_DECODE, bros.BROS_BF16, batch.num_seqs, batch.num_q_heads,
                                        batch.head_dim, max_ctx)
    assert 0 < wsb <= (48 << 20)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    ref_out = torch.full_like(dev.q_decode, float("nan"))
    bros.bros_attn_decode(ref_out, dev.q_decode, dev.k_pool, dev.v_pool, dev.block_tables, dev.dir, dev.cls,
                          dev.ctx_lens, max_ctx, workspace=ws)
    out = torch.full_like(dev.q_decode, float("nan"))
    _noalloc_via_c_abi(bros, out, dev, max_ctx)
    torch.cuda.synchronize()
    return bros.to_host_bits(out), bros.to_host_bits(ref_out)


def test_noalloc_decode_matches_the_workspace_entry_point_twice():
    # First call: long contexts cut between many workers (partials and merge
    # in the scratch array); second call: a smaller batch, which must not see
    # the first call's leftovers.
    rng = np.random.default_rng(31)
    big_ctx = rng.integers(1024, 8000, 48)
    big = W.custom(big_ctx, [W.BE if i % 3 else W.RT for i in range(48)], 32, 8, seed=31, spare_blocks=13)
    small = W.custom([7000, 33, 2500, 16, 9], [W.BE, W.RT, W.BE, W.RT, W.BE], 32, 8, seed=32)
    for name, b in (("first, 48 rows", big), ("second, 5 rows", small)):
        announce(f"decode_noalloc {name} sum_ctx={int(b.ctx_lens.sum())}")
        got, ref_gpu = _both(b)
        assert np.array_equal(got, ref_gpu), f"{name}: noalloc output differs from bros_attn_decode"
        ref = oracle.decode(b.q_decode, b.k_pool, b.v_pool, b.block_tables, b.dir, b.ctx_lens, b.dtype)
        compare(got, ref, "bf16", f"noalloc {name}")
