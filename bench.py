#!/usr/bin/env python3
"""Benchmark of one mixed RT/BE paged-attention step on one MI355X.

A step is the whole hot path over one synthetic batch whose KV lives in one
shared bidirectional pool: bros_kv_write of the step's new tokens, then
bros_attn_prefill_chunk for the RT prefill chunks, then bros_attn_decode for
the BE decode rows. Default workload: llama3-8b-mixed-step (4 RT chunks of 512
new tokens on c0 ~ U{0..2048} cached tokens, 128 BE decode rows with ctx ~
U{512..8192}, 32 q / 8 KV heads, head_dim 128, bf16, 40000-block pool).

Timing: inputs resident in HBM; W untimed warm-up steps, then timed passes of
exactly K steps each, every pass between two synchronizations: one that
brackets every call with HIP events (the per-call figures), one with HIP
events around the decode call on the stream it runs on and, recorded by the
library, around the decode kernel inside it (the roofline's launch duration),
the headline pass, with HIP events only around the K steps (an
event inside a step costs it a few microseconds), and the per-call pass again.
The GPU's clocks ramp up over the first ~30 steps after it has been idle
(10-step batches right after start: 440, 424, 418, then 416 us), so the
headline and roofline passes run on a GPU that has been busy for the pass
before them, and the per-call figures are the second per-call pass's (the
first one's are in per_call_us_first_pass). Then R single steps, each
after a scrub that reads and writes 1 GiB outside its events, give the median,
p10 and p90 of a step whose KV comes from HBM. Prints ONE JSON line:
  value     = algorithmic bytes of a step / step time (GB/s, whole job)
  roofline  = the dominant kernel (the decode kernel): the decode's algorithmic
              bytes per launch / that kernel's average duration between HIP
              events the library records around it on its stream, against 8
              TB/s HBM; call_frac is the same over the whole decode call
              (kernel and merge, events around the call in the per-call pass)
  scrubbed  = p10 / p50 / p90 of the scrubbed single steps
  cpu_baseline = the CPU oracle timed on one host core over one whole step
              (or, when the pools do not fit in float64, a sample of rows).
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
BF16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak, published
METRIC = "µs per mixed RT/BE attention step + achieved KV GB/s (% of HBM peak)"
# The oracle runs one whole step when both pools widened to float64 fit in this many bytes.
FP64_POOL_LIMIT = 16e9
# Bytes the scrub between timed repetitions reads and writes (4x the 256 MiB last-level cache).
SCRUB_BYTES = 1 << 30

# HBM traffic of the decode kernel from rocprofv3 counters (FETCH_SIZE and WRITE_SIZE, one
# counter per run, KiB per dispatch of decode_mfma_kernel).
# The counters are scaled by what they read for a plain 1 GiB device copy
# (--calibrate-copy): FETCH_SIZE reads half the bytes copied, WRITE_SIZE all of them.
FETCH_SCALE = 2.0
WRITE_SCALE = 1.0
DECODE_SOURCES = ("paper_2504_09590_amd/csrc/decode.hip", "paper_2504_09590_amd/csrc/decode_device.h",
                  "paper_2504_09590_amd/csrc/decode_common.h",
                  "paper_2504_09590_amd/csrc/bros_device.h",
                  "paper_2504_09590_amd/csrc/bros_kernels.h")
DECODE_COUNTERS = {
    # workload: (sha256 of DECODE_SOURCES when the counters were read, FETCH_SIZE KiB, WRITE_SIZE KiB)
    "llama3-70b-decode": ("f12efb5159ca9ddbc4bd03e7871364d4a41b058062ac265b93f1a6bc2576ee52", 4991849.4, 16514.1),
    "llama3-8b-decode": ("f12efb5159ca9ddbc4bd03e7871364d4a41b058062ac265b93f1a6bc2576ee52", 454831.8, 5197.5),
    "llama3-8b-mixed-step": ("f12efb5159ca9ddbc4bd03e7871364d4a41b058062ac265b93f1a6bc2576ee52", 1129273.9, 6173.5),
    "llama3-8b-pressure": ("f12efb5159ca9ddbc4bd03e7871364d4a41b058062ac265b93f1a6bc2576ee52", 601668.8, 10115.7),
}


def decode_sources_sha256() -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in DECODE_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def decode_traffic(workload: str):
    """Counter-measured HBM bytes per decode call, or None when no counters were read for
    this workload or the decode sources changed since they were."""
    rec = DECODE_COUNTERS.get(workload)
    if rec is None or rec[0] != decode_sources_sha256():
        return None
    return int(round((rec[1] * FETCH_SCALE + rec[2] * WRITE_SCALE) * 1024))


def algorithmic_work(batch):
    """Bytes and flops the method must move / do for one step, per call."""
    e = batch.elem_bytes
    hkv, hq, d = batch.num_kv_heads, batch.num_q_heads, batch.head_dim
    P = batch.num_prefill
    kv_tok = 2 * hkv * d * e                         # K + V bytes of one token
    ctx = batch.ctx_lens.astype(np.int64)
    dec_rows = batch.num_seqs - P
    dec_kv = int(ctx[P:].sum()) * kv_tok
    dec_qo = 2 * dec_rows * hq * d * e
    dec_tables = int(((ctx[P:] + 15) // 16).sum()) * 4 + dec_rows * (4 + 1)
    pre_kv = int(ctx[:P].sum()) * kv_tok             # each chunk reads its context once
    tq = int(batch.cu_q[-1])
    pre_qo = 2 * tq * hq * d * e
    n = np.diff(batch.cu_q).astype(np.int64)
    c0 = ctx[:P] - n
    # causal flops: QK^T and PV, 2 flops per MAC each
    pre_flops = int(sum(4 * hq * d * int(np.sum(c0[i] + np.arange(1, n[i] + 1))) for i in range(P)))
    tn = int(batch.cu_new[-1])
    write_bytes = 2 * tn * kv_tok                    # read the new rows, write them into the pool
    return {
        "kv_write": {"bytes": write_bytes},
        "prefill": {"bytes": pre_kv + pre_qo, "flops": pre_flops},
        "decode": {"bytes": dec_kv + dec_qo + dec_tables, "kv_bytes": dec_kv},
        "step_bytes": write_bytes + pre_kv + pre_qo + dec_kv + dec_qo + dec_tables,
    }


def cpu_baseline(batch, budget_s: float, step_bytes: int):
    """The oracle, as it stands, timed on one host core (BLAS limited to one
    thread). When the pools fit in float64 within FP64_POOL_LIMIT, it runs one
    whole step of the workload: kv_write, prefill_chunk over every chunk and
    decode over every row, one oracle call each on the same inputs (each call
    widens the whole pool once). Otherwise it runs decode rows in batch order,
    each on a pool cut to that row's blocks, until `budget_s` is spent, and the
    rate is scaled to the step. Returns GB/s of algorithmic bytes and seconds
    per step."""
    import oracle
    from threadpoolctl import threadpool_limits

    from paper_2504_09590_amd import workload
    P = batch.num_prefill
    kv_tok = 2 * batch.num_kv_heads * batch.head_dim * batch.elem_bytes
    whole = 2 * batch.k_pool.size * 8 <= FP64_POOL_LIMIT
    with threadpool_limits(1):
        t0 = time.perf_counter()
        if whole:
            k1, v1 = oracle.kv_write(batch.k_pool, batch.v_pool, batch.k_new, batch.v_new, batch.block_tables,
                                     batch.dir, batch.pos0, batch.cu_new)
            if P:
                oracle.prefill_chunk(batch.q_prefill, batch.cu_q, k1, v1, batch.block_tables[:P], batch.dir[:P],
                                     batch.ctx_lens[:P], batch.dtype)
            if batch.num_seqs > P:
                oracle.decode(batch.q_decode, k1, v1, batch.block_tables[P:], batch.dir[P:], batch.ctx_lens[P:],
                              batch.dtype)
            dt = time.perf_counter() - t0
            per_step = dt
            sample = (f"whole step: kv_write of {int(batch.cu_new[-1])} tokens, {P} prefill chunks, "
                      f"{batch.num_seqs - P} decode rows; {dt:.1f} s fp64 NumPy on one core")
        else:
            done, rows = 0, 0
            for r in range(batch.num_seqs - P):
                if time.perf_counter() - t0 > budget_s:
                    break
                s = P + r
                tab, kp, vp = workload.compact_pool(batch.block_tables[s:s + 1], batch.ctx_lens[s:s + 1],
                                                    batch.k_pool, batch.v_pool)
                oracle.decode(batch.q_decode[r:r + 1], kp, vp, tab, batch.dir[s:s + 1], batch.ctx_lens[s:s + 1],
                              batch.dtype)
                done += int(batch.ctx_lens[s]) * kv_tok
                rows += 1
            dt = time.perf_counter() - t0
            per_step = dt * step_bytes / max(done, 1)
            sample = (f"{rows} of {batch.num_seqs - P} decode rows in batch order, each on a pool cut to its "
                      f"blocks; {dt:.1f} s fp64 NumPy on one core, scaled to the step")
    return {"value": round(step_bytes / per_step / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": sample, "seconds_per_step": round(per_step, 2), "seconds": round(dt, 2)}


def swap_figures(step, per_call, K):
    """Lazy-checkpoint figures: the gather/scatter kernels inside the step, and
    the host copies of the same rows (copy engine) timed alone, K of each."""
    import torch
    lane, n = step.swap, int(step.swap_ids.numel())
    moved = 2 * lane._bytes(n)                                       # K and V, each way
    rates = {}
    for name in ("d2h", "h2d"):
        cs = (lane.out_stream if name == "d2h" else lane.in_stream) or torch.cuda.current_stream()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(cs)
        for _ in range(K):
            if name == "d2h":
                lane.copy_out(step.host_out_k, step.host_out_v, n, cs)
            else:
                lane.copy_in(step.host_in_k, step.host_in_v, n, cs)
        b.record(cs)
        torch.cuda.synchronize()
        us = a.elapsed_time(b) / K * 1e3
        rates[name] = {"us": round(us, 2), "GB/s": round(moved / (us * 1e-6) / 1e9, 1)}
    in_step = {}
    for kind in ("d2h", "h2d"):
        us = [a.elapsed_time(b) * 1e3 for k, a, b in lane.timing if k == kind]
        if us:
            in_step[kind] = {"us": round(float(np.mean(us)), 2), "GB/s": round(moved / (np.mean(us) * 1e-6) / 1e9, 1)}
    lane.timing = None
    g, sc = per_call["swap_gather"] * 1e3, per_call["swap_scatter"] * 1e3
    return {"slots": n, "bytes_each_way": moved,
            "gather_us": round(g, 2), "scatter_us": round(sc, 2),
            "gather_hbm_GBps": round(2 * moved / (g * 1e-6) / 1e9, 1),
            "scatter_hbm_GBps": round(2 * moved / (sc * 1e-6) / 1e9, 1),
            "copies_in_step": in_step, "copies_alone": rates}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="llama3-8b-mixed-step")
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--overlap", action="store_true", help="run the prefill on a side stream beside the decode")
    ap.add_argument("--prefill-cus", type=int, default=0,
                    help="run the prefill on the first N compute units and the write and decode on the rest "
                         "(N a multiple of 32; implies --overlap)")
    ap.add_argument("--swap-serial", action="store_true",
                    help="with --swap-slots: enqueue the host copies on the step's stream between its kernels")
    ap.add_argument("--swap-slots", type=int, default=0,
                    help="also checkpoint and restore N slots per step (lazy checkpointing), the host copies "
                         "overlapping the attention")
    ap.add_argument("--fused", action="store_true",
                    help="run the prefill and the decode in one launch (bros_attn_mixed) instead of two calls")
    ap.add_argument("--reps", type=int, default=50,
                    help="single steps timed one by one after a cache scrub each (median, p10, p90)")
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of oracle work for cpu_baseline when the whole step does not fit in memory")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device copy K times (scales FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU; --gpus {args.gpus} is not supported "
              "(the step shards by KV head or by sequence with no exchange, but only the one-GPU path is built)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    if args.calibrate_copy:
        n = 1 << 28                                   # 2^28 fp32 = 1 GiB read + 1 GiB written per copy
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "device copy", "bytes_read_per_launch": 4 * n,
                          "bytes_written_per_launch": 4 * n, "launches": args.steps}), flush=True)
        return

    from paper_2504_09590_amd import bros, workload
    from paper_2504_09590_amd.step import MixedStep

    batch = workload.generate(args.workload, seed=args.seed)
    bros.bros_check_batch(batch.block_tables, batch.dir, batch.cls, batch.ctx_lens, batch.num_blocks)
    dev = bros.to_device(batch)
    step = MixedStep(batch, dev, overlap=args.overlap, prefill_cus=args.prefill_cus, swap_slots=args.swap_slots,
                     swap_serial=args.swap_serial, fused=args.fused)
    work = algorithmic_work(batch)
    stream = step.main if step.main is not None else torch.cuda.current_stream()

    for _ in range(args.warmup):
        step.run()
    torch.cuda.synchronize()

    K = args.steps
    side = step.side if step.overlap else stream
    main_call = "mixed" if step.fused else "decode"   # the dominant call, bracketed for the roofline

    def timed_steps(bracket: str):
        """K steps between two events on `stream`. bracket "none": no other
        event (the headline pass; each event in the stream costs a step a few
        microseconds); "main": the dominant call bracketed by events of its own
        (the roofline's launch duration); "all": every call, for the per-call
        breakdown."""
        names = ("kv_write",) + (("mixed",) if step.fused else ("prefill", "decode")) + \
            (("swap_gather", "swap_scatter") if step.swap else ())
        chosen = {"none": (), "main": (main_call,), "all": names}[bracket]
        ev = {k: [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
              for k in chosen}
        written = [torch.cuda.Event() for _ in range(K)]
        prefilled = [torch.cuda.Event() for _ in range(K)]
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

        # the decode kernel alone, apart from its merge: events the library
        # records around that kernel inside the bracketed decode call
        kev = None
        if bracket == "main" and main_call == "decode" and batch.dtype == "bf16":
            kev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
            for a, b in kev:   # (a torch event exists once it has been recorded)
                a.record(stream); b.record(stream)

        def call(name, i, s, fn):
            if name in ev:
                a, b = ev[name][i]
                a.record(s)
                if kev is not None and name == "decode":
                    bros.bros_set_decode_kernel_events(*kev[i])
                    fn(s)
                    bros.bros_set_decode_kernel_events(None, None)
                else:
                    fn(s)
                b.record(s)
            else:
                fn(s)

        if step.swap:
            step.swap.timing = [] if bracket == "all" else None
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        start.record(stream)
        for i in range(K):
            # one step: kv_write, then prefill (on the side stream when overlapping) and decode
            if step.swap:
                call("swap_gather", i, stream, step.swap_out)
            call("kv_write", i, stream, step.kv_write)
            if step.swap:
                call("swap_scatter", i, stream, step.swap_in)
            if step.overlap:
                written[i].record(stream)
                side.wait_event(written[i])
            if step.fused:
                call("mixed", i, stream, step.mixed)
            else:
                call("prefill", i, side, step.prefill)
                call("decode", i, stream, step.decode)
            if step.overlap:
                prefilled[i].record(side)
                stream.wait_event(prefilled[i])
            if step.swap:
                step.swap_next(stream)
        end.record(stream)
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t0) * 1e3
        per = {k: float(np.mean([a.elapsed_time(b) for a, b in pairs])) for k, pairs in ev.items()}
        if kev is not None:
            per["decode_kernel"] = float(np.mean([a.elapsed_time(b) for a, b in kev]))
        return start.elapsed_time(end) / K, per, wall

    def scrubbed_reps(R: int):
        """R single steps, each preceded (outside its events) by a scrub that
        reads and writes SCRUB_BYTES, so that no KV of the previous step is
        left in the last-level cache. Returns the step times in ms."""
        scrub = torch.zeros(SCRUB_BYTES // 4, dtype=torch.float32, device=dev.k_pool.device)
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(R)]
        torch.cuda.synchronize()
        with torch.cuda.stream(stream):
            for a, b in ev:
                scrub.add_(1.0)
                a.record(stream)
                if step.swap:
                    step.swap_out(stream)
                step.kv_write(stream)
                if step.swap:
                    step.swap_in(stream)
                if step.overlap:
                    a2 = torch.cuda.Event()
                    a2.record(stream)
                    side.wait_event(a2)
                if step.fused:
                    step.mixed(stream)
                else:
                    step.prefill(side)
                    step.decode(stream)
                if step.overlap:
                    b2 = torch.cuda.Event()
                    b2.record(side)
                    stream.wait_event(b2)
                if step.swap:
                    step.swap_next(stream)
                b.record(stream)
        torch.cuda.synchronize()
        del scrub
        return np.array([a.elapsed_time(b) for a, b in ev])

    # the headline pass (no event inside a step), a pass with the dominant
    # call bracketed, a pass with every call bracketed, then single steps with
    # a cache scrub before each
    # the headline pass after two others: the clocks have ramped up by then (see the
    # docstring); the pass that brackets every call runs first and again last, and
    # its figures come from the second run
    _, per_call_first, _ = timed_steps("all")
    ms_main, per_main, _ = timed_steps("main")
    ms, _, wall_ms = timed_steps("none")
    ms_inst, per_call, _ = timed_steps("all")
    if "decode_kernel" in per_main:
        per_call["decode_kernel"] = per_main["decode_kernel"]   # the roofline pass: the kernel alone
    else:
        per_call[main_call + "_alone_bracketed"] = per_main[main_call]
    reps = scrubbed_reps(max(args.reps, 1))

    call_ms = per_main.get(main_call)
    # the whole call as the per-call pass times it (no event between its kernels)
    call_alone_ms = per_call.get(main_call, call_ms)
    roof = None
    if call_ms:
        if step.fused:
            nbytes = work["decode"]["bytes"] + work["prefill"]["bytes"]
            kernel, traffic, dec_ms = "bros_attn_mixed (mixed_kernel + decode_mfma_merge_kernel)", None, call_ms
        elif "decode_kernel" in per_main:
            # the dominant kernel on its own; the whole call (kernel + merge) beside it
            nbytes = work["decode"]["bytes"]
            kernel, dec_ms = "decode_mfma_kernel", per_main["decode_kernel"]
            traffic = decode_traffic(batch.name)
        else:
            nbytes = work["decode"]["bytes"]
            kernel, traffic, dec_ms = "bros_attn_decode (decode kernel + merge)", None, call_ms
        achieved = nbytes / (dec_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic, "kernel": kernel,
                "bytes_per_launch": nbytes, "avg_launch_us": round(dec_ms * 1e3, 2),
                "call_avg_us": round(call_alone_ms * 1e3, 2),
                "call_frac": round(nbytes / (call_alone_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}

    value = work["step_bytes"] / (ms * 1e-3) / 1e9
    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "GB/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "us_per_step": round(ms * 1e3, 2),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": batch.dtype,
        "data": "synthetic", "hbm_frac_step": round(value / HBM_PEAK_GBS, 4),
        "config": {"workload": batch.name, "seed": batch.seed, "num_seqs": batch.num_seqs,
                   "prefill_chunks": batch.num_prefill, "decode_rows": batch.num_seqs - batch.num_prefill,
                   "q_heads": batch.num_q_heads, "kv_heads": batch.num_kv_heads, "head_dim": batch.head_dim,
                   "block_size": 16, "pool_blocks": batch.num_blocks, "sum_ctx": int(batch.ctx_lens.sum()),
                   "overlap": bool(step.overlap), "prefill_cus": step.prefill_cus,
                   "swap_slots": args.swap_slots,
                   "swap_serial": bool(args.swap_serial), "fused": bool(step.fused)},
        "per_call_us": {k: round(v * 1e3, 2) for k, v in per_call.items()},
        "per_call_us_first_pass": {k: round(v * 1e3, 2) for k, v in per_call_first.items()},
        "us_per_step_main_call_timed": round(ms_main * 1e3, 2),
        "us_per_step_every_call_timed": round(ms_inst * 1e3, 2),
        "scrubbed": {"scrub": True, "scrub_bytes": SCRUB_BYTES, "reps": int(reps.size),
                     "us_p10": round(float(np.percentile(reps, 10)) * 1e3, 2),
                     "us_p50": round(float(np.percentile(reps, 50)) * 1e3, 2),
                     "us_p90": round(float(np.percentile(reps, 90)) * 1e3, 2)},
        "step_bytes": work["step_bytes"],
        "roofline": roof,
        "wall_ms_timed_region": round(wall_ms, 3),
    }
    if per_call.get("prefill"):
        tf = work["prefill"]["flops"] / (per_call["prefill"] * 1e-3) / 1e12
        line["prefill_mfma"] = {"achieved_tflops": round(tf, 1), "peak_tflops": BF16_MFMA_PEAK_TFLOPS,
                                "frac": round(tf / BF16_MFMA_PEAK_TFLOPS, 4), "flops": work["prefill"]["flops"]}
    if step.swap:
        line["swap"] = swap_figures(step, per_call, K)
    step.close()
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(batch, args.cpu_budget, work["step_bytes"])
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
