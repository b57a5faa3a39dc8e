"""The oracle's decode output for every row of a generated workload.

Started by the GPU tests as a child process that never touches the GPU:

    python -m tests.oracle_rows CONFIG OUT.npy [--workers N]

It regenerates workload CONFIG from its seed, splits the decode rows into
groups and runs oracle.decode on each group in forked worker processes. Each
group gets a pool of only the blocks its rows reference
(workload.compact_pool), so each worker widens only those blocks to float64;
the oracle itself is called as it stands. The float64 result [rows][Hq][D] is
saved to OUT.npy.
"""

from __future__ import annotations

import argparse
import multiprocessing as mp
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2504_09590_amd import workload as W  # noqa: E402

_BATCH = None   # the workload, inherited by the forked workers


def _decode_rows(rows):
    from threadpoolctl import threadpool_limits
    b = _BATCH
    P = b.num_prefill
    tab, kp, vp = W.compact_pool(b.block_tables[P:][rows], b.ctx_lens[P:][rows], b.k_pool, b.v_pool)
    with threadpool_limits(1):   # one core per worker process
        return oracle.decode(b.q_decode[rows], kp, vp, tab, b.dir[P:][rows], b.ctx_lens[P:][rows], b.dtype)


def decode_all_rows(batch, workers: int) -> np.ndarray:
    """oracle.decode over every decode row of `batch`, in groups on `workers` processes."""
    global _BATCH
    _BATCH = batch
    P = batch.num_prefill
    n = batch.num_seqs - P
    order = np.argsort(-batch.ctx_lens[P:].astype(np.int64), kind="stable")
    n_groups = max(1, min(n, 4 * workers))
    groups = [np.sort(order[i::n_groups]) for i in range(n_groups)]
    with mp.get_context("fork").Pool(workers) as pool:
        parts = pool.map(_decode_rows, groups, chunksize=1)
    out = np.zeros((n, batch.num_q_heads, batch.head_dim), dtype=np.float64)
    for g, part in zip(groups, parts):
        out[g] = part
    return out


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("config", type=int)
    ap.add_argument("out")
    ap.add_argument("--workers", type=int, default=min(16, len(os.sched_getaffinity(0))))
    args = ap.parse_args()
    t0 = time.perf_counter()
    batch = W.generate(args.config)
    print(f"[oracle_rows] {batch.name}: generated in {time.perf_counter() - t0:.1f} s", flush=True)
    t1 = time.perf_counter()
    out = decode_all_rows(batch, args.workers)
    np.save(args.out, out)
    print(f"[oracle_rows] {batch.name}: {out.shape[0]} rows on {args.workers} processes in "
          f"{time.perf_counter() - t1:.1f} s", flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
