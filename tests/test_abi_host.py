"""Host-side checks of the C ABI (no GPU needed): the library loads and exports
every symbol include/bros_attn.h declares, argument validation rejects bad
calls before anything is launched, the workspace query is consistent, and the
batch checker agrees with the oracle's independent slot-ownership count."""

import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2504_09590_amd import workload as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bros_attn.h")

bros = pytest.importorskip("paper_2504_09590_amd.bros", reason="libbros_attn.so not built")

FAKE = 1 << 20   # a 16-byte aligned non-NULL address; only used on paths rejected before launch


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bros_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_three_entry_points():
    names = declared_functions()
    for fn in ("bros_kv_write", "bros_attn_decode", "bros_attn_prefill_chunk"):
        assert fn in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(bros.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing
    assert sorted(bros.EXPORTED) == declared_functions()


def test_status_strings_and_version():
    for code, name in bros.STATUS.items():
        assert bros.LIB.bros_status_str(code).decode() == name
    assert bros.LIB.bros_abi_version() == 9


# --- argument validation (returns before any HIP call) -----------------------

def _decode(**kw):
    args = dict(out=FAKE, q=FAKE, k=FAKE, v=FAKE, nb=10, bt=FAKE, maxb=4, dir=FAKE, cls=None, dpe=0,
                ctx=FAKE, max_ctx=64, S=2, hq=8, hkv=2, d=128, bs=16, scale=0.0, dtype=1,
                ws=None, wsb=0, stream=None)
    args.update(kw)
    return bros.LIB.bros_attn_decode(args["out"], args["q"], args["k"], args["v"], args["nb"], args["bt"],
                                     args["maxb"], args["dir"], args["cls"], args["dpe"], args["ctx"], args["max_ctx"],
                                     args["S"], args["hq"], args["hkv"], args["d"], args["bs"], args["scale"],
                                     args["dtype"], args["ws"], args["wsb"], args["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=7), -3),
    (dict(d=64), -4),
    (dict(bs=32), -4),
    (dict(hq=6, hkv=4), -2),
    (dict(hq=48, hkv=2), -4),          # group 24
    (dict(out=None), -1),
    (dict(bt=None), -1),
    (dict(dir=None, cls=None), -1),
    (dict(dpe=2), -2),                 # direction mode neither per sequence nor per entry
    (dict(dir=None, cls=FAKE, dpe=1), -1),   # a direction table needs dir
    (dict(S=-1), -2),
    (dict(nb=0), -2),
    (dict(maxb=0), -2),
    (dict(out=FAKE + 4), -2),          # misaligned
    (dict(max_ctx=100000), -5),        # needs a split-K workspace
])
def test_decode_rejects(kw, code):
    assert _decode(**kw) == code
    assert bros.LIB.bros_last_error().decode() != ""


def test_decode_with_no_sequences_is_a_noop():
    assert _decode(S=0, out=None, q=None) == 0


def test_kv_write_rejects():
    L = bros.LIB
    args = [FAKE, FAKE, 5, FAKE, FAKE, 10, FAKE, 4, FAKE, None, 0, FAKE, FAKE, 2, 2, 128, 16, 1, None]
    a = list(args); a[17] = 9
    assert L.bros_kv_write(*a) == -3
    a = list(args); a[13] = 0
    assert L.bros_kv_write(*a) == -2
    a = list(args); a[11] = None
    assert L.bros_kv_write(*a) == -1
    a = list(args); a[10] = 3
    assert L.bros_kv_write(*a) == -2         # direction mode
    a = list(args); a[2] = 0
    assert L.bros_kv_write(*a) == 0          # no tokens: no-op
    a = list(args); a[14] = 16385
    assert L.bros_kv_write(*a) == -4         # more KV heads than the kernel's index split covers


def test_prefill_rejects():
    L = bros.LIB
    base = [FAKE, FAKE, FAKE, 64, 32, FAKE, FAKE, 10, FAKE, 4, FAKE, None, 0, FAKE, 64, 2, 8, 2, 128, 16,
            0.0, 1, None, 0, None]
    a = list(base); a[4] = 0
    assert L.bros_attn_prefill_chunk(*a) == -2
    a = list(base); a[2] = None
    assert L.bros_attn_prefill_chunk(*a) == -1
    a = list(base); a[10] = None; a[11] = FAKE; a[12] = 1   # a direction table needs dir
    assert L.bros_attn_prefill_chunk(*a) == -1
    a = list(base); a[21] = 0; a[14] = 100000   # fp32 path needs a workspace
    assert L.bros_attn_prefill_chunk(*a) == -5
    a = list(base); a[3] = 0
    assert L.bros_attn_prefill_chunk(*a) == 0


@pytest.mark.parametrize("fn", ["bros_kv_gather", "bros_kv_scatter"])
def test_kv_move_rejects(fn):
    L = getattr(bros.LIB, fn)
    if fn == "bros_kv_gather":   # k_pool, v_pool, nb, ids, n, k_out, v_out, hkv, d, bs, dtype, stream
        base = [FAKE, FAKE, 10, FAKE, 5, FAKE, FAKE, 8, 128, 16, 1, None]
        idx = dict(nb=2, ids=3, n=4, hkv=7, d=8, bs=9, dtype=10, ptr=5)
    else:                        # k_in, v_in, ids, n, k_pool, v_pool, nb, hkv, d, bs, dtype, stream
        base = [FAKE, FAKE, FAKE, 5, FAKE, FAKE, 10, 8, 128, 16, 1, None]
        idx = dict(nb=6, ids=2, n=3, hkv=7, d=8, bs=9, dtype=10, ptr=0)
    for key, val, code in (("dtype", 7, -3), ("bs", 8, -4), ("d", 64, -4), ("hkv", 0, -2), ("n", -1, -2),
                           ("nb", 0, -2), ("ids", None, -1), ("ptr", None, -1), ("ptr", FAKE + 4, -2)):
        a = list(base)
        a[idx[key]] = val
        assert L(*a) == code, (key, val)
    a = list(base)
    a[idx["n"]] = 0
    a[idx["ids"]] = None
    assert L(*a) == 0               # nothing to move: no-op


def test_copy_dma_rejects_null_and_allows_empty():
    assert bros.LIB.bros_copy_dma(None, FAKE, 16, None) == -1
    assert bros.LIB.bros_copy_dma(FAKE, None, 16, None) == -1
    assert bros.LIB.bros_copy_dma(None, None, 0, None) == 0


def test_check_slot_ids():
    ok = np.array([5, 3, 159, -1, -1, 160, 160, 0], dtype=np.int32)   # repeats only outside the pool
    bros.bros_check_slot_ids(ok, 10)
    with pytest.raises(bros.BrosError, match="slot id 3"):
        bros.bros_check_slot_ids(np.array([1, 3, 2, 3], dtype=np.int32), 10)
    assert bros.LIB.bros_check_slot_ids(None, 0, 10) == 0
    assert bros.LIB.bros_check_slot_ids(None, 2, 10) == -1
    assert bros.LIB.bros_check_slot_ids(None, 2, 0) == -2


@pytest.mark.parametrize("first,num", [(0, 0), (0, 48), (16, 32), (-32, 64), (0, -32)])
def test_cu_share_rejects_uneven_ranges(first, num):
    out = ctypes.c_void_p(123)
    assert bros.LIB.bros_stream_create_cu_share(first, num, ctypes.byref(out)) == -2
    assert out.value is None
    assert "multiples of 32" in bros.LIB.bros_last_error().decode()


def test_cu_share_rejects_null_outputs():
    assert bros.LIB.bros_stream_create_cu_share(0, 32, None) == -1
    assert bros.LIB.bros_stream_destroy(None) == -1


def test_workspace_query():
    q = bros.bros_attn_workspace_size
    assert q(0, 0, 4, 8, 128, 64) == 0              # fp32, single split: no workspace
    assert q(0, 0, 64, 32, 128, 8192) > 0           # fp32, several splits
    small = q(0, 1, 4, 8, 128, 64)                  # bf16: row prefix + per-worker partials, any length
    big = q(0, 1, 64, 32, 128, 8192)
    assert 0 < small < big and big % 16 == 0
    assert q(0, 1, 64, 32, 128, 16384) == big       # bf16 size does not grow with the context
    assert q(0, 1, 65, 32, 128, 8192) > big
    # bf16 prefill on the matrix cores: the optional split workspace, one size for every call
    split = q(1, 1, 2048, 32, 128, 8192)
    assert split > 0 and split % 16 == 0 and split == q(1, 1, 16, 8, 128, 32768)
    assert q(1, 1, 2048, 32, 128, 32769) != split   # beyond 32768: the vector path's own size
    assert q(1, 0, 2048, 32, 128, 8192) > 0
    assert q(0, 1, 4, 8, 64, 64) == 0               # unsupported head_dim


# --- the batch checker -------------------------------------------------------

@pytest.mark.parametrize("config", [1, 2, 3, 4, 5])
def test_checker_accepts_generated_batches(config):
    b = W.generate(config, with_pool=False)
    bros.bros_check_batch(b.block_tables, b.dir, b.cls, b.ctx_lens, b.num_blocks)
    bros.bros_check_batch(b.block_tables, None, b.cls, b.ctx_lens, b.num_blocks)


def _tiny():
    tables = np.array([[2, 0], [3, 0], [1, -1]], dtype=np.int32)
    return tables, np.array([1, -1, 1], dtype=np.int8), np.array([21, 27, 16], dtype=np.int32)


def test_checker_accepts_full_shared_block():
    t, d, c = _tiny()
    bros.bros_check_batch(t, d, None, c, 4)


@pytest.mark.parametrize("mutate,needle", [
    (lambda t, d, c: c.__setitem__(1, 28), "already owned"),       # 5 + 12 > 16 slots
    (lambda t, d, c: t.__setitem__((0, 1), 4), "outside"),
    (lambda t, d, c: t.__setitem__((0, 0), -3), "outside"),
    (lambda t, d, c: d.__setitem__(0, 0), "direction"),
    (lambda t, d, c: c.__setitem__(2, 33), "exceeds"),
    (lambda t, d, c: c.__setitem__(2, 17), "outside"),             # reaches the -1 pad
    (lambda t, d, c: c.__setitem__(2, -1), "negative"),
    (lambda t, d, c: d.__setitem__(1, 1), "already owned"),        # both from the left
])
def test_checker_rejects(mutate, needle):
    t, d, c = _tiny()
    mutate(t, d, c)
    with pytest.raises(bros.BrosError) as ei:
        bros.bros_check_batch(t, d, None, c, 4)
    assert ei.value.status == -7 and needle in str(ei.value)


@pytest.mark.parametrize("config", [1, 2, 3, 5])
def test_checker_accepts_direction_tables(config):
    """The paper's per-entry direction table (Sec. 6): flipping entries of
    blocks a sequence fills keeps the batch consistent, and the checker agrees
    with the oracle's slot-ownership count."""
    from tests.gpu_helpers import with_direction_table
    b = with_direction_table(W.generate(config), frac=0.5, seed=config)
    assert b.dir.ndim == 2
    assert oracle.slot_owner_counts(b.block_tables, b.dir, b.ctx_lens, b.num_blocks).max() <= 1
    bros.bros_check_batch(b.block_tables, b.dir, None, b.ctx_lens, b.num_blocks)


def test_checker_rejects_bad_direction_tables():
    # RT tail (5 slots from the left) and BE tail (11 from the right) share block 0
    t = np.array([[2, 0], [3, 0]], dtype=np.int32)
    c = np.array([21, 27], dtype=np.int32)
    d = np.array([[1, 1], [-1, -1]], dtype=np.int8)
    bros.bros_check_batch(t, d, None, c, 4)
    bad = d.copy()
    bad[0, 1] = -1                       # the RT tail walked from the right collides with the BE tail
    with pytest.raises(bros.BrosError, match="already owned"):
        bros.bros_check_batch(t, bad, None, c, 4)
    assert oracle.slot_owner_counts(t, bad, c, 4).max() == 2
    bad = d.copy()
    bad[1, 0] = 0                        # not a direction
    with pytest.raises(bros.BrosError, match="entry 0"):
        bros.bros_check_batch(t, bad, None, c, 4)
    with pytest.raises(ValueError):
        bros.bros_check_batch(t, d[:, :1], None, c, 4)   # table shape must match


def test_checker_rejects_unsupported_block_size():
    t, d, c = _tiny()
    with pytest.raises(bros.BrosError) as ei:
        bros.bros_check_batch(t, d, None, c, 4, block_size=8)
    assert ei.value.status == -4


def test_checker_agrees_with_oracle_on_random_batches():
    rng = np.random.default_rng(3)
    for trial in range(200):
        S = int(rng.integers(1, 6))
        nb = int(rng.integers(1, 8))
        maxb = int(rng.integers(1, 4))
        tables = rng.integers(0, nb, size=(S, maxb)).astype(np.int32)
        dirs = rng.choice([1, -1], size=S).astype(np.int8)
        ctx = rng.integers(0, maxb * 16 + 1, size=S).astype(np.int32)
        counts = oracle.slot_owner_counts(tables, dirs, ctx, nb)
        expect_ok = counts.max(initial=0) <= 1
        try:
            bros.bros_check_batch(tables, dirs, None, ctx, nb)
            got_ok = True
        except bros.BrosError:
            got_ok = False
        assert got_ok == expect_ok, (trial, tables, dirs, ctx)


def test_noalloc_decode_rejects_a_batch_beyond_its_scratch_array():
    # Checked before any HIP call: 4096 rows x 32 heads need more workspace
    # than the static array holds (NULL tensors are never reached).
    need = bros.bros_attn_workspace_size(bros.BROS_WS_DECODE, bros.BROS_BF16, 4096, 32, 128, 8192)
    assert need > (48 << 20)
    st = bros.LIB.bros_attn_decode_noalloc(None, None, None, None, 10, None, 4, None, None, 0, None, 8192, 4096,
                                           32, 8, 128, 16, 0.0, bros.BROS_BF16, None)
    assert st == -5
    msg = bros.LIB.bros_last_error().decode()
    assert "scratch" in msg and str(need) in msg
    # within the limit the size check passes and the usual argument checks answer
    st = bros.LIB.bros_attn_decode_noalloc(None, None, None, None, 10, None, 4, None, None, 0, None, 64, 2,
                                           32, 8, 128, 16, 0.0, bros.BROS_BF16, None)
    assert st == -1


def test_slot_ids_follow_the_oracle_mapping():
    # The library's slot ids of (sequence, position) pairs equal the oracle's
    # own (block, slot) mapping, per-sequence and per-entry directions alike.
    b = W.custom([40, 17, 70, 9, 33], [W.RT, W.BE, W.BE, W.RT, W.RT], 8, 4, seed=41, spare_blocks=5)
    rng = np.random.default_rng(41)
    seqs = rng.integers(0, b.num_seqs, 200)
    pos = np.array([rng.integers(0, b.ctx_lens[s]) for s in seqs])
    for dirs in (b.dir, np.where(rng.random(b.block_tables.shape) < 0.5, 1, -1).astype(np.int8)):
        got = bros.bros_slot_ids(b.block_tables, dirs, b.cls, b.num_blocks, seqs, pos)
        for i, (s, p) in enumerate(zip(seqs, pos)):
            blk, slot = oracle.physical_location(b.block_tables, dirs, int(s), [int(p)])
            assert got[i] == int(blk[0]) * 16 + int(slot[0])
    # direction from the class when dir is NULL
    got = bros.bros_slot_ids(b.block_tables, None, b.cls, b.num_blocks, seqs, pos)
    assert np.array_equal(got, bros.bros_slot_ids(b.block_tables, b.dir, None, b.num_blocks, seqs, pos))
    with pytest.raises(bros.BrosError, match="outside"):
        bros.bros_slot_ids(b.block_tables, b.dir, b.cls, b.num_blocks, [b.num_seqs], [0])
    with pytest.raises(bros.BrosError, match="beyond"):
        bros.bros_slot_ids(b.block_tables, b.dir, b.cls, b.num_blocks, [0], [16 * b.block_tables.shape[1]])


def test_decode_kernel_events_hook_takes_both_or_neither():
    L = bros.LIB
    assert L.bros_set_decode_kernel_events(FAKE, None) == -1
    assert L.bros_set_decode_kernel_events(None, FAKE) == -1
    assert L.bros_set_decode_kernel_events(None, None) == 0
