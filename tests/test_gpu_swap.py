"""Lazy-checkpoint gather/scatter (bros_kv_gather / bros_kv_scatter) against the
oracle, bit for bit: several workgroups plus a ragged tail, ids outside the
pool, an empty list, a pinned host destination, and the Sec. 5.2 scenario
(checkpoint, overwrite by the peer, restore into a fresh block) run through
the GPU kernels, where the peer's decode must come out bit-identical."""

import json
import os

import numpy as np
import pytest

import oracle
from tests.gpu_helpers import announce, compare, require_gpu

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _random(rng, shape, dtype):
    if dtype == "bf16":
        return rng.integers(0, 1 << 16, size=shape, dtype=np.uint16) & np.uint16(0xBFFF)
    return rng.standard_normal(shape).astype(np.float32)


def _to_dev(torch, x, dtype):
    t = torch.from_numpy(np.ascontiguousarray(x).view(np.int16) if dtype == "bf16" else np.ascontiguousarray(x))
    t = t.cuda()
    return t.view(torch.bfloat16) if dtype == "bf16" else t


def _to_host(t, dtype):
    import torch
    if dtype == "bf16":
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def _ids(rng, nb, n, extra_outside=True):
    ids = rng.permutation(nb * 16)[:n].astype(np.int32)
    if extra_outside and n > 40:
        ids[[7, 19, 33]] = [-1, nb * 16, np.iinfo(np.int32).max]
    return ids


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n", [1, 37, 1003])
def test_gather_matches_oracle(dtype, n):
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    rng = np.random.default_rng(100 + n)
    nb, hkv, d = 300, 8, 128
    kp, vp = _random(rng, (nb, hkv, 16, d), dtype), _random(rng, (nb, hkv, 16, d), dtype)
    ids = _ids(rng, nb, n)
    announce(f"kv_gather {dtype} n={n}")
    k_dev, v_dev = _to_dev(torch, kp, dtype), _to_dev(torch, vp, dtype)
    k_out = torch.full((n, hkv, d), 7, dtype=k_dev.dtype, device="cuda")
    v_out = torch.full((n, hkv, d), 7, dtype=k_dev.dtype, device="cuda")
    bros.bros_kv_gather(k_dev, v_dev, torch.from_numpy(ids).cuda(), k_out, v_out)
    torch.cuda.synchronize()
    assert np.array_equal(_to_host(k_out, dtype), oracle.kv_gather(kp, ids))
    assert np.array_equal(_to_host(v_out, dtype), oracle.kv_gather(vp, ids))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n", [1, 37, 1003])
def test_scatter_matches_oracle(dtype, n):
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    rng = np.random.default_rng(200 + n)
    nb, hkv, d = 300, 8, 128
    kp, vp = _random(rng, (nb, hkv, 16, d), dtype), _random(rng, (nb, hkv, 16, d), dtype)
    kr, vr = _random(rng, (n, hkv, d), dtype), _random(rng, (n, hkv, d), dtype)
    ids = _ids(rng, nb, n)
    bros.bros_check_slot_ids(ids, nb)
    announce(f"kv_scatter {dtype} n={n}")
    k_dev, v_dev = _to_dev(torch, kp, dtype), _to_dev(torch, vp, dtype)
    bros.bros_kv_scatter(_to_dev(torch, kr, dtype), _to_dev(torch, vr, dtype), torch.from_numpy(ids).cuda(),
                         k_dev, v_dev)
    torch.cuda.synchronize()
    assert np.array_equal(_to_host(k_dev, dtype), oracle.kv_scatter(kp, kr, ids))
    assert np.array_equal(_to_host(v_dev, dtype), oracle.kv_scatter(vp, vr, ids))


def test_empty_list_moves_nothing():
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    kp = torch.zeros((4, 2, 16, 128), dtype=torch.bfloat16, device="cuda")
    ids = torch.zeros((0,), dtype=torch.int32, device="cuda")
    out = torch.zeros((0, 2, 128), dtype=torch.bfloat16, device="cuda")
    announce("kv_gather/kv_scatter empty")
    bros.bros_kv_gather(kp, kp, ids, out, out)
    bros.bros_kv_scatter(out, out, ids, kp, kp)
    torch.cuda.synchronize()
    assert not kp.any()


def test_gather_into_pinned_host_memory():
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    rng = np.random.default_rng(3)
    nb, hkv, d, n = 64, 8, 128, 200
    kp, vp = _random(rng, (nb, hkv, 16, d), "bf16"), _random(rng, (nb, hkv, 16, d), "bf16")
    ids = _ids(rng, nb, n)
    k_host = torch.empty((n, hkv, d), dtype=torch.bfloat16, pin_memory=True)
    v_host = torch.empty((n, hkv, d), dtype=torch.bfloat16, pin_memory=True)
    announce("kv_gather to pinned host")
    bros.bros_kv_gather(_to_dev(torch, kp, "bf16"), _to_dev(torch, vp, "bf16"), torch.from_numpy(ids).cuda(),
                        k_host, v_host)
    torch.cuda.synchronize()
    assert np.array_equal(k_host.view(torch.int16).numpy().view(np.uint16), oracle.kv_gather(kp, ids))
    assert np.array_equal(v_host.view(torch.int16).numpy().view(np.uint16), oracle.kv_gather(vp, ids))


def test_lazy_checkpoint_scenario_on_gpu():
    """The hand-enumerated Sec. 5.2 scenario through the kernels: the peer's
    decode after checkpoint, overwrite and restore is bit-identical to its
    decode before, and matches the oracle."""
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    with open(os.path.join(ROOT, "tests", "golden", "lazy_checkpoint.json")) as f:
        g = json.load(f)
    rng = np.random.default_rng(17)
    nb, hkv, hq, d = g["num_blocks"], 8, 32, 128
    B, a = g["before"]["B"], g["before"]["a"]
    tables = np.zeros((2, 2), dtype=np.int32)
    tables[0] = B["block_table"]
    tables[1, 0] = a["block_table"][0]
    dirs = np.array([B["dir"], a["dir"]], dtype=np.int8)
    ctx = np.array([B["ctx"], a["ctx"]], dtype=np.int32)
    kp, vp = _random(rng, (nb, hkv, 16, d), "bf16"), _random(rng, (nb, hkv, 16, d), "bf16")
    q = _random(rng, (2, hq, d), "bf16")
    k_dev, v_dev = _to_dev(torch, kp, "bf16"), _to_dev(torch, vp, "bf16")
    q_dev = _to_dev(torch, q, "bf16")
    out = torch.empty_like(q_dev)
    ws = torch.empty(bros.bros_attn_workspace_size(bros.BROS_WS_DECODE, bros.BROS_BF16, 2, hq, d, 64),
                     dtype=torch.uint8, device="cuda")

    def decode(tab, c):
        bros.bros_attn_decode(out, q_dev, k_dev, v_dev, torch.from_numpy(tab).cuda(), torch.from_numpy(dirs).cuda(),
                              None, torch.from_numpy(c).cuda(), int(c.max()), workspace=ws)
        torch.cuda.synchronize()
        return _to_host(out, "bf16")[1].copy()

    announce("lazy checkpoint scenario: decode before")
    before = decode(tables, ctx)
    compare(before[None], oracle.decode(q, kp, vp, tables, dirs, ctx, "bf16", seqs=[1])[1:2], "bf16", "before")

    # checkpoint the victims into pinned host memory (via a device staging buffer)
    victims = oracle.overwritten_peer_tokens(tables, dirs, ctx, 0, g["write"]["positions"])
    ids = np.array(g["checkpoint_slot_ids"], dtype=np.int32)
    n = len(ids)
    stage_k = torch.empty((n, hkv, d), dtype=torch.bfloat16, device="cuda")
    stage_v = torch.empty_like(stage_k)
    announce("lazy checkpoint scenario: gather victims")
    bros.bros_kv_gather(k_dev, v_dev, torch.from_numpy(ids).cuda(), stage_k, stage_v)
    host_k = torch.empty(stage_k.shape, dtype=torch.bfloat16, pin_memory=True)
    host_v = torch.empty(stage_v.shape, dtype=torch.bfloat16, pin_memory=True)
    host_k.copy_(stage_k, non_blocking=True)
    host_v.copy_(stage_v, non_blocking=True)

    # the writer overwrites them
    k_new, v_new = _random(rng, (n, hkv, d), "bf16"), _random(rng, (n, hkv, d), "bf16")
    announce("lazy checkpoint scenario: kv_write")
    bros.bros_kv_write(_to_dev(torch, k_new, "bf16"), _to_dev(torch, v_new, "bf16"), k_dev, v_dev,
                       torch.from_numpy(tables).cuda(), torch.from_numpy(dirs).cuda(), None,
                       torch.tensor([g["write"]["positions"][0], 0], dtype=torch.int32, device="cuda"),
                       torch.tensor([0, n, n], dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    ctx_after = ctx.copy()
    ctx_after[0] += n
    assert not np.array_equal(decode(tables, ctx_after), before)

    # restore: a's entry 0 moves to a fresh block
    r = g["restore"]
    new_tables = tables.copy()
    new_tables[1, r["table_entry"]] = r["new_block"]
    lost = {v[1] for v in victims}
    keep = np.array([p for p in range(int(ctx[1])) if p not in lost])
    src = oracle.slot_ids(*oracle.physical_location(tables, dirs, 1, keep))
    dst = oracle.slot_ids(*oracle.physical_location(new_tables, dirs, 1, keep))
    back = oracle.slot_ids(*oracle.physical_location(new_tables, dirs, 1, np.array(sorted(lost))))
    mk = torch.empty((len(keep), hkv, d), dtype=torch.bfloat16, device="cuda")
    mv = torch.empty_like(mk)
    announce("lazy checkpoint scenario: restore")
    bros.bros_kv_gather(k_dev, v_dev, torch.from_numpy(src).cuda(), mk, mv)
    bros.bros_kv_scatter(mk, mv, torch.from_numpy(dst).cuda(), k_dev, v_dev)
    rk, rv = host_k.cuda(non_blocking=True), host_v.cuda(non_blocking=True)
    bros.bros_kv_scatter(rk, rv, torch.from_numpy(back).cuda(), k_dev, v_dev)
    after = decode(new_tables, ctx_after)
    assert np.array_equal(after, before)


def test_copy_dma_round_trip_through_pinned_host():
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    rng = np.random.default_rng(9)
    rows = _random(rng, (777, 8, 128), "bf16")
    src = _to_dev(torch, rows, "bf16")
    host = torch.empty(src.shape, dtype=torch.bfloat16, pin_memory=True)
    back = torch.zeros_like(src)
    side = torch.cuda.Stream()
    announce("bros_copy_dma device -> pinned host -> device")
    torch.cuda.synchronize()
    bros.bros_copy_dma(host, src, stream=side)
    bros.bros_copy_dma(back, host, stream=side)
    torch.cuda.synchronize()
    assert np.array_equal(host.view(torch.int16).numpy().view(np.uint16), rows)
    assert np.array_equal(_to_host(back, "bf16"), rows)


def test_copy_dma_is_ordered_on_its_stream():
    """Fresh data each round: a kernel writes it, the copy engine takes it to
    pinned host memory and back into a device buffer, and a kernel on the same
    stream reads that buffer right after. 64 MiB each way takes over a
    millisecond on the engine, so a stream that did not wait for the copy
    would read the previous round's values."""
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    n = 16 << 20                                              # int32 words: 64 MiB
    s = torch.cuda.Stream()
    host = torch.empty(n, dtype=torch.int32, pin_memory=True)
    dev_in = torch.zeros(n, dtype=torch.int32, device="cuda")
    src = torch.empty(n, dtype=torch.int32, device="cuda")
    base = torch.arange(n, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    for r in range(6):
        announce(f"bros_copy_dma ordering round {r}")
        with torch.cuda.stream(s):
            torch.add(base, r * 7919, out=src)                    # the kernel that writes the data
            bros.bros_copy_dma(host, src, stream=s)
            bros.bros_copy_dma(dev_in, host, stream=s)
            got = dev_in.clone()                                  # the kernel that reads it
        s.synchronize()
        assert torch.equal(got, base + r * 7919), f"round {r}: the stream read before the copy landed"
        assert torch.equal(host, torch.arange(n, dtype=torch.int32) + r * 7919)


def test_copy_dma_both_directions_on_two_streams():
    """One stream copies out while another copies in; each result matches."""
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    n = 8 << 20
    a, b = torch.cuda.Stream(), torch.cuda.Stream()
    src = torch.randint(-2**31, 2**31 - 1, (n,), dtype=torch.int32, device="cuda")
    host_in = torch.randint(-2**31, 2**31 - 1, (n,), dtype=torch.int32).pin_memory()
    host_out = torch.empty(n, dtype=torch.int32, pin_memory=True)
    dst = torch.empty(n, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    announce("bros_copy_dma both directions at once")
    for _ in range(3):
        bros.bros_copy_dma(host_out, src, stream=a)
        bros.bros_copy_dma(dst, host_in, stream=b)
    torch.cuda.synchronize()
    assert torch.equal(host_out, src.cpu())
    assert torch.equal(dst.cpu(), host_in)


def test_copy_dma_refuses_pageable_host_memory():
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    src = torch.zeros(1024, dtype=torch.int32, device="cuda")
    pageable = torch.zeros(1024, dtype=torch.int32)
    host = torch.zeros(1024, dtype=torch.int32, pin_memory=True)
    torch.cuda.synchronize()
    assert bros.LIB.bros_copy_dma(ctypes_ptr(pageable), ctypes_ptr(src), 4096, None) == -2
    assert bros.LIB.bros_copy_dma(ctypes_ptr(pageable), ctypes_ptr(host), 4096, None) == -2


def ctypes_ptr(t):
    import ctypes
    return ctypes.c_void_p(t.data_ptr())


def test_copy_dma_refuses_a_capturing_stream():
    """An engine copy is issued when requested, so it cannot be part of a
    graph: under capture the call is refused and nothing is recorded."""
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    src = torch.zeros(1024, dtype=torch.int32, device="cuda")
    host = torch.zeros(1024, dtype=torch.int32, pin_memory=True)
    out = torch.zeros(1024, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    with torch.cuda.graph(g, stream=s):
        rc = bros.LIB.bros_copy_dma(ctypes_ptr(host), ctypes_ptr(src), 4096, ctypes_ptr_stream(s))
        out.add_(1)
    assert rc == -4
    g.replay()
    torch.cuda.synchronize()
    assert int(out[0]) == 1


def ctypes_ptr_stream(s):
    import ctypes
    return ctypes.c_void_p(s.cuda_stream)
