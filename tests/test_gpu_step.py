"""One whole mixed step (kv_write -> prefill -> decode) through MixedStep, the
dispatch the benchmark times, on the full mixed-step workload, against the
oracle's step; with and without the prefill on a side stream, and with the
two halves on disjoint compute-unit shares (which also checks that the decode
grid fits a share)."""

import numpy as np
import pytest

import oracle
from paper_2504_09590_amd import workload as W
from tests.gpu_helpers import announce, compare, oracle_step, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mixed():
    b = W.generate(3)
    return b, oracle_step(b)


@pytest.mark.parametrize("overlap,prefill_cus,swap_slots",
                         [(False, 0, 0), (True, 0, 0), (True, 64, 0), (True, 224, 0), (False, 0, 1024),
                          (True, 64, 1024), (False, 0, -1024)])
def test_mixed_step_full(mixed, overlap, prefill_cus, swap_slots):
    serial = swap_slots < 0          # a negative count: the serial arrangement
    swap_slots = abs(swap_slots)
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    from paper_2504_09590_amd.step import MixedStep
    b, (k1, v1, pre_ref, dec_ref) = mixed
    dev = bros.to_device(b)
    announce(f"mixed step {b.name} overlap={overlap} prefill_cus={prefill_cus} swap_slots={swap_slots} "
             f"serial={serial}")
    step = MixedStep(b, dev, overlap=overlap, prefill_cus=prefill_cus, swap_slots=swap_slots, swap_serial=serial)
    pre, dec = step.run()
    if swap_slots:   # a second step restores what the first checkpointed
        pre, dec = step.run()
    torch.cuda.synchronize()
    if swap_slots:
        ids = step.swap_ids.cpu().numpy()
        assert np.array_equal(bros.to_host_bits(step.host_out_k), oracle.kv_gather(k1, ids))
        assert np.array_equal(bros.to_host_bits(step.host_out_v), oracle.kv_gather(v1, ids))
    step.close()
    for name, ref, got in (("k", k1, dev.k_pool), ("v", v1, dev.v_pool)):
        assert np.array_equal(bros.to_host_bits(got), ref), f"{name} pool after the step"
    mx_p, mean_p = compare(bros.to_host_bits(pre), pre_ref, "bf16", "step prefill")
    mx_d, mean_d = compare(bros.to_host_bits(dec), dec_ref, "bf16", "step decode")
    print(f"step prefill max {mx_p:.3g} mean {mean_p:.3g}; decode max {mx_d:.3g} mean {mean_d:.3g}")


def test_mixed_step_replays_from_a_hip_graph(mixed):
    """The whole step (write, prefill, decode) captured once in a HIP graph and
    replayed: every replay, with eager work and synchronisations between them,
    gives the eager step's outputs bit for bit (the kernels allocate nothing
    and clear nothing with memset, so a serving loop can capture them)."""
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    from paper_2504_09590_amd.step import MixedStep
    b, (k1, v1, pre_ref, dec_ref) = mixed
    dev = bros.to_device(b)
    announce(f"mixed step {b.name} captured in a HIP graph")
    step = MixedStep(b, dev)
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        pre, dec = step.run()       # eager, also warms the library's per-device queries
        side.synchronize()
        eager = (bros.to_host_bits(pre).copy(), bros.to_host_bits(dec).copy())
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=side):
            step.run()
    for i in range(3):
        scratch = torch.randn(1 << 20, device="cuda")     # eager work between the replays
        pre.fill_(float("nan"))
        dec.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert float(scratch.abs().sum()) > 0
        assert np.array_equal(bros.to_host_bits(pre), eager[0]), f"prefill, replay {i}"
        assert np.array_equal(bros.to_host_bits(dec), eager[1]), f"decode, replay {i}"
    step.close()
    compare(eager[0], pre_ref, "bf16", "step prefill (eager)")
    compare(eager[1], dec_ref, "bf16", "step decode (eager)")
    for name, ref, got in (("k", k1, dev.k_pool), ("v", v1, dev.v_pool)):
        assert np.array_equal(bros.to_host_bits(got), ref), f"{name} pool after the replays"


@pytest.mark.parametrize("fused", [False, True])
def test_table_entries_past_the_context_are_never_used(fused):
    """Entries at index >= ceil(ctx / 16) of a block table are not the
    sequence's (the ABI ignores them): filled with garbage (out-of-range ids,
    negative ids, other sequences' blocks), the step gives the same pools and
    outputs as the oracle's step on the clean tables."""
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    from paper_2504_09590_amd.step import MixedStep
    from tests.gpu_helpers import poison_unowned
    ctx = [64 + 130, 45, 2000, 700, 31, 17, 400]
    cls = [W.RT, W.RT, W.BE, W.RT, W.BE, W.BE, W.RT]
    new = [130, 45, 1, 1, 1, 1, 1]
    b = W.custom(ctx, cls, 32, 8, seed=71, num_prefill=2, new_counts=new, spare_blocks=6)
    poison_unowned(b)
    ref = oracle_step(b)
    rng = np.random.default_rng(71)
    garbage = np.array([2**31 - 1, -2**31, -1, -7, b.num_blocks, b.num_blocks + 5, 0, 3], dtype=np.int64)
    nblk = (b.ctx_lens.astype(np.int64) + 15) // 16
    for s in range(b.num_seqs):
        tail = b.block_tables[s, nblk[s]:]
        tail[:] = rng.choice(garbage, size=tail.shape).astype(np.int32)
    announce(f"step with garbage past each table's context, fused={fused}")
    dev = bros.to_device(b)
    step = MixedStep(b, dev, fused=fused)
    pre, dec = step.run()
    torch.cuda.synchronize()
    step.close()
    k1, v1, pre_ref, dec_ref = ref
    for name, r, got in (("k", k1, dev.k_pool), ("v", v1, dev.v_pool)):
        assert np.array_equal(bros.to_host_bits(got), r), f"{name} pool after the step"
    compare(bros.to_host_bits(pre), pre_ref, "bf16", "prefill with garbage table tails")
    compare(bros.to_host_bits(dec), dec_ref, "bf16", "decode with garbage table tails")
