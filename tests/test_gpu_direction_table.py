"""The paper's per-entry direction table (Sec. 6: one flag per block-table
entry, shaped like the tables) through every kernel, against the oracle: a
random half of the entries whose block a sequence fills are walked the other
way, so a wrong entry lookup moves keys between slots and fails parity. Also:
a table that repeats the per-sequence flags gives bit-identical results to
the per-sequence form."""

import dataclasses

import numpy as np
import pytest

from paper_2504_09590_amd import workload as W
from tests.gpu_helpers import announce, compare, oracle_step, require_gpu, with_direction_table
from tests.test_gpu_decode import ref_decode, run_decode

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("config", [1, 2, 5])
def test_decode_with_direction_table(config):
    b = with_direction_table(W.generate(config), frac=0.5, seed=config)
    announce(f"decode {b.name} with a direction table")
    compare(run_decode(b), ref_decode(b), b.dtype, f"{b.name} direction table")


def test_mixed_step_with_direction_table():
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    from paper_2504_09590_amd.step import MixedStep
    b = with_direction_table(W.generate(3), frac=0.5, seed=3)
    k1, v1, pre_ref, dec_ref = oracle_step(b)
    dev = bros.to_device(b)
    announce("mixed step with a direction table")
    step = MixedStep(b, dev)
    pre, dec = step.run()
    torch.cuda.synchronize()
    assert np.array_equal(bros.to_host_bits(dev.k_pool), k1)
    assert np.array_equal(bros.to_host_bits(dev.v_pool), v1)
    compare(bros.to_host_bits(pre), pre_ref, "bf16", "prefill, direction table")
    compare(bros.to_host_bits(dec), dec_ref, "bf16", "decode, direction table")


def test_repeated_flags_match_per_sequence_form():
    require_gpu()
    b = W.generate(2)
    tab = dataclasses.replace(b, dir=np.ascontiguousarray(np.repeat(b.dir[:, None], b.block_tables.shape[1], axis=1)))
    announce("decode: direction table repeating the per-sequence flags")
    assert np.array_equal(run_decode(b), run_decode(tab))
