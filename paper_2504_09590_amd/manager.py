"""ctypes binding of the host block manager and the Alg. 1 scheduler
(csrc/manager.cpp, declared in include/bros_attn.h). Marshalling only.

Sec. 5.2: FindBlock / FindPreemptBlock, lazy checkpointing and the preemption
table; Sec. 4.2: the priority-based packing algorithm and adaptive batch
sizing. A grow or restore returns a Plan: the peer tokens to checkpoint before
the write (victims), device moves of relocated entries, destinations of
restored tokens, and the slot of every new token.
"""

from __future__ import annotations

import ctypes
from dataclasses import dataclass

import numpy as np

I32P = ctypes.POINTER(ctypes.c_int32)


class _Plan(ctypes.Structure):
    _fields_ = [("victims", I32P), ("victims_cap", ctypes.c_int32), ("num_victims", ctypes.c_int32),
                ("move_src", I32P), ("move_dst", I32P), ("moves_cap", ctypes.c_int32), ("num_moves", ctypes.c_int32),
                ("restore_pos", I32P), ("restore_dst", I32P), ("restores_cap", ctypes.c_int32),
                ("num_restores", ctypes.c_int32),
                ("written_pos", I32P), ("written_slot", I32P), ("written_cap", ctypes.c_int32),
                ("num_written", ctypes.c_int32)]


class SchedReq(ctypes.Structure):
    _fields_ = [("id", ctypes.c_int32), ("prefill", ctypes.c_int32), ("n_new", ctypes.c_int32),
                ("ctx_after", ctypes.c_int32), ("remaining_us", ctypes.c_double), ("m_cpu", ctypes.c_int32)]


# The same record as a numpy structured type, for building queues without a
# Python loop (layout checked against ctypes at import).
SCHED_DTYPE = np.dtype([("id", "<i4"), ("prefill", "<i4"), ("n_new", "<i4"), ("ctx_after", "<i4"),
                        ("remaining_us", "<f8"), ("m_cpu", "<i4")], align=True)
assert SCHED_DTYPE.itemsize == ctypes.sizeof(SchedReq)


class CostModelC(ctypes.Structure):
    _fields_ = [("coef", (ctypes.c_double * 3) * 2), ("per_request", ctypes.c_int32)]


def declare(lib) -> None:
    P, I = ctypes.c_void_p, ctypes.c_int32
    sig = {
        "bros_mgr_create": ([I], P), "bros_mgr_destroy": ([P], None),
        "bros_mgr_add_request": ([P, I, I], ctypes.c_int), "bros_mgr_release": ([P, I], ctypes.c_int),
        "bros_mgr_grow": ([P, I, I, ctypes.POINTER(_Plan)], ctypes.c_int),
        "bros_mgr_restore": ([P, I, ctypes.POINTER(_Plan)], ctypes.c_int),
        "bros_mgr_query": ([P, I, I32P, I32P, I32P], ctypes.c_int),
        "bros_mgr_table": ([P, I, I32P, I], ctypes.c_int),
        "bros_mgr_free_blocks": ([P], I), "bros_mgr_validate": ([P], ctypes.c_int), "bros_mgr_available": ([P, I], I),
        "bros_mgr_entries_needed": ([P, I, I], I), "bros_mgr_preemption_table": ([P, I32P, I], I),
        "bros_schedule": ([P, ctypes.POINTER(SchedReq), I, ctypes.POINTER(SchedReq), I, I,
                           ctypes.POINTER(CostModelC), I32P, I32P, I32P, I32P, I32P], ctypes.c_int),
        "bros_next_batch_size": ([I, I, I, I], I),
        "bros_mgr_grow_batch": ([P, I32P, I32P, I, I, ctypes.POINTER(_Plan), I32P, I32P], ctypes.c_int),
        "bros_mgr_plan_bound": ([P, I32P, I32P, I], I),
        "bros_schedule_pulled": ([P, ctypes.POINTER(SchedReq), I, ctypes.POINTER(SchedReq), I,
                                  ctypes.POINTER(SchedReq), I, I, ctypes.POINTER(CostModelC), I32P, I32P, I32P,
                                  I32P, I32P], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res


def _lib():
    from . import bros
    return bros


@dataclass
class Plan:
    victims: np.ndarray       # [n][4] request, position, block, slot
    move_src: np.ndarray      # slot ids
    move_dst: np.ndarray
    restore_pos: np.ndarray   # positions of the request
    restore_dst: np.ndarray   # slot ids
    written_pos: np.ndarray
    written_slot: np.ndarray


class BlockManager:
    def __init__(self, num_blocks: int):
        b = _lib()
        self._b = b
        self.num_blocks = int(num_blocks)
        self.h = b.LIB.bros_mgr_create(self.num_blocks)
        if not self.h:
            raise b.BrosError(-2, b.LIB.bros_last_error().decode())

    def close(self):
        if self.h:
            self._b.LIB.bros_mgr_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def add(self, req: int, cls: int):
        self._b._check(self._b.LIB.bros_mgr_add_request(self.h, int(req), int(cls)))

    def release(self, req: int):
        self._b._check(self._b.LIB.bros_mgr_release(self.h, int(req)))

    def _buffers(self, cap: int):
        """Plan buffers of at least `cap` entries, kept between calls."""
        if getattr(self, "_cap", 0) < cap:
            self._cap = max(cap, 2 * getattr(self, "_cap", 0))
            self._bufs = {k: np.zeros(self._cap * (4 if k == "victims" else 1), dtype=np.int32)
                          for k in ("victims", "move_src", "move_dst", "restore_pos", "restore_dst", "written_pos",
                                    "written_slot")}
            ptr = {k: v.ctypes.data_as(I32P) for k, v in self._bufs.items()}
            self._plan = _Plan(ptr["victims"], self._cap, 0, ptr["move_src"], ptr["move_dst"], self._cap, 0,
                               ptr["restore_pos"], ptr["restore_dst"], self._cap, 0, ptr["written_pos"],
                               ptr["written_slot"], self._cap, 0)
        return self._bufs, self._plan

    def _run(self, fn, *args, cap: int) -> Plan:
        # caps are upper bounds by construction (a new token victimises at most
        # one peer token, a moved entry holds at most 15 tokens), so a call
        # never fails for want of room after changing the manager
        bufs, plan = self._buffers(cap)
        st = fn(self.h, *args, ctypes.byref(plan))
        out = Plan(bufs["victims"][:4 * plan.num_victims].reshape(-1, 4).copy(),
                   bufs["move_src"][:plan.num_moves].copy(), bufs["move_dst"][:plan.num_moves].copy(),
                   bufs["restore_pos"][:plan.num_restores].copy(), bufs["restore_dst"][:plan.num_restores].copy(),
                   bufs["written_pos"][:plan.num_written].copy(), bufs["written_slot"][:plan.num_written].copy())
        if st != 0:
            # what happened before the failure stays done: the caller applies it
            err = self._b.BrosError(st, self._b.LIB.bros_last_error().decode())
            err.plan = out
            raise err
        return out

    def grow(self, req: int, n_new: int) -> Plan:
        return self._run(self._b.LIB.bros_mgr_grow, int(req), int(n_new), cap=max(64, 2 * int(n_new) + 64))

    def grow_batch(self, reqs, n_new, restore_first: bool = True):
        """One call for an iteration's block management (restore, then grow,
        per request, in order). Returns (plan, ends, status): the concatenated
        plan, the [n][4] running counts of victims, moves, restores and
        written tokens after each request, and each request's status. A
        failing request raises nothing here: its status says so."""
        r = np.ascontiguousarray(reqs, dtype=np.int32)
        k = np.ascontiguousarray(n_new, dtype=np.int32)
        n = int(r.shape[0])
        ends = np.zeros((max(n, 1), 4), dtype=np.int32)
        status = np.zeros(max(n, 1), dtype=np.int32)
        cap = int(self._b.LIB.bros_mgr_plan_bound(self.h, r.ctypes.data_as(I32P), k.ctypes.data_as(I32P), n))
        if cap < 0:
            raise self._b.BrosError(-2, "bros_mgr_plan_bound: an unknown request or a negative count")
        bufs, plan = self._buffers(cap)
        st = self._b.LIB.bros_mgr_grow_batch(self.h, r.ctypes.data_as(I32P), k.ctypes.data_as(I32P), n,
                                             1 if restore_first else 0, ctypes.byref(plan),
                                             ends.ctypes.data_as(I32P), status.ctypes.data_as(I32P))
        if st not in (0, -7, -8):
            self._b._check(st)
        out = Plan(bufs["victims"][:4 * plan.num_victims].reshape(-1, 4).copy(),
                   bufs["move_src"][:plan.num_moves].copy(), bufs["move_dst"][:plan.num_moves].copy(),
                   bufs["restore_pos"][:plan.num_restores].copy(), bufs["restore_dst"][:plan.num_restores].copy(),
                   bufs["written_pos"][:plan.num_written].copy(), bufs["written_slot"][:plan.num_written].copy())
        return out, ends[:n].copy(), status[:n].copy()

    def restore(self, req: int) -> Plan:
        ctx, _, ck = self.query(req)
        return self._run(self._b.LIB.bros_mgr_restore, int(req), cap=max(64, ctx + 64))

    def query(self, req: int):
        a, b, c = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        self._b._check(self._b.LIB.bros_mgr_query(self.h, int(req), ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)))
        return a.value, b.value, c.value        # ctx, entries, checkpointed tokens

    def table(self, req: int) -> np.ndarray:
        _, n, _ = self.query(req)
        out = np.zeros(max(n, 1), dtype=np.int32)
        self._b._check(self._b.LIB.bros_mgr_table(self.h, int(req), out.ctypes.data_as(I32P), len(out)))
        return out[:n]

    def validate(self):
        self._b._check(self._b.LIB.bros_mgr_validate(self.h))

    def free_blocks(self) -> int:
        return int(self._b.LIB.bros_mgr_free_blocks(self.h))

    def available(self, cls: int) -> int:
        return int(self._b.LIB.bros_mgr_available(self.h, int(cls)))

    def preemption_table(self) -> np.ndarray:
        n = int(self._b.LIB.bros_mgr_preemption_table(self.h, None, 0))
        out = np.zeros((max(n, 1), 3), dtype=np.int32)
        self._b.LIB.bros_mgr_preemption_table(self.h, out.ctypes.data_as(I32P), n)
        return out[:n]


def schedule(mgr: BlockManager, rt, be, batch_size: int, coef, per_request: bool = False):
    """Alg. 1. rt / be: sequences of dicts with id, prefill, n_new, ctx_after,
    remaining_us (RT) / m_cpu (BE), or numpy arrays of SCHED_DTYPE. coef: ((a0, a1, b) prefill, (a0, a1, b)
    decode). Returns (rt ids, be ids, over_budget)."""
    b = mgr._b

    def pack(reqs):
        if isinstance(reqs, np.ndarray):
            arr = np.ascontiguousarray(reqs, dtype=SCHED_DTYPE)
        else:
            arr = np.zeros(max(len(reqs), 1), dtype=SCHED_DTYPE)
            for i, r in enumerate(reqs):
                arr[i] = (int(r["id"]), int(r.get("prefill", 0)), int(r["n_new"]), int(r["ctx_after"]),
                          float(r.get("remaining_us", 0.0)), int(r.get("m_cpu", 0)))
        return arr.ctypes.data_as(ctypes.POINTER(SchedReq)), arr

    cm = CostModelC()
    for ph in range(2):
        for k in range(3):
            cm.coef[ph][k] = float(coef[ph][k])
    cm.per_request = 1 if per_request else 0
    out_rt = np.zeros(max(len(rt), 1), dtype=np.int32)
    out_be = np.zeros(max(len(be), 1), dtype=np.int32)
    n_rt, n_be, over = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    (prt, _keep_rt), (pbe, _keep_be) = pack(rt), pack(be)
    b._check(b.LIB.bros_schedule(mgr.h, prt, len(rt), pbe, len(be), int(batch_size), ctypes.byref(cm),
                                 out_rt.ctypes.data_as(I32P), ctypes.byref(n_rt), out_be.ctypes.data_as(I32P),
                                 ctypes.byref(n_be), ctypes.byref(over)))
    return out_rt[:n_rt.value].tolist(), out_be[:n_be.value].tolist(), bool(over.value)


def schedule_pulled(mgr: BlockManager, pending, waiting, be, batch_size: int, coef, per_request: bool = False):
    """Alg. 1 with the request-pulling optimization (Sec. 4.2): pending RT
    requests in any order, waiting RT requests in ascending remaining time,
    BE requests. Arrays of SCHED_DTYPE. Returns (rt ids, be ids, over_budget)."""
    b = mgr._b
    arrs = [np.ascontiguousarray(q if len(q) else np.zeros(1, dtype=SCHED_DTYPE), dtype=SCHED_DTYPE)
            for q in (pending, waiting, be)]
    ptrs = [a.ctypes.data_as(ctypes.POINTER(SchedReq)) for a in arrs]
    cm = CostModelC()
    for ph in range(2):
        for k in range(3):
            cm.coef[ph][k] = float(coef[ph][k])
    cm.per_request = 1 if per_request else 0
    out_rt = np.zeros(max(len(pending) + len(waiting), 1), dtype=np.int32)
    out_be = np.zeros(max(len(be), 1), dtype=np.int32)
    n_rt, n_be, over = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    b._check(b.LIB.bros_schedule_pulled(mgr.h, ptrs[0], len(pending), ptrs[1], len(waiting), ptrs[2], len(be),
                                        int(batch_size), ctypes.byref(cm), out_rt.ctypes.data_as(I32P),
                                        ctypes.byref(n_rt), out_be.ctypes.data_as(I32P), ctypes.byref(n_be),
                                        ctypes.byref(over)))
    return out_rt[:n_rt.value].tolist(), out_be[:n_be.value].tolist(), bool(over.value)


def next_batch_size(current: int, base: int, max_size: int, over_budget: bool) -> int:
    return int(_lib().LIB.bros_next_batch_size(int(current), int(base), int(max_size), 1 if over_budget else 0))


def main(argv=None):
    """Host cost of one iteration's scheduling and block management on one CPU
    thread: Alg. 1 over every queued request, then one decode token for every
    scheduled request (restores, FindBlock / FindPreemptBlock, lazy
    checkpoints). Two arrangements: one C call per request with a full sort of
    the RT queue (per_request), and the iteration's block management in one
    batched C call with Sec. 4.2's request pulling (batched; the waiting RT
    queue is kept in ascending remaining time and only the pending queue is
    sorted)."""
    import argparse
    import json
    import time
    ap = argparse.ArgumentParser(description=main.__doc__)
    ap.add_argument("--requests", type=int, default=512)
    ap.add_argument("--blocks", type=int, default=40000)
    ap.add_argument("--iterations", type=int, default=200)
    ap.add_argument("--batch", type=int, default=256)
    ap.add_argument("--seed", type=int, default=0)
    args = ap.parse_args(argv)
    from .costmodel import load_fitted
    fitted = load_fitted()   # the per-request form fitted on this library's kernels (us)
    coef = (tuple(fitted.coef["prefill/per_request"]), tuple(fitted.coef["decode/per_request"]))
    out = {"requests": args.requests, "blocks": args.blocks, "batch": args.batch, "iterations": args.iterations}
    for mode in ("per_request", "batched"):
        rng = np.random.default_rng(args.seed)
        mgr = BlockManager(args.blocks)
        cls = {}
        for rid in range(1, args.requests + 1):
            c = 0 if rng.random() < 0.25 else 1
            mgr.add(rid, c)
            cls[rid] = c
            try:
                mgr.grow(rid, int(rng.integers(64, 1200)))
            except Exception:
                mgr.release(rid)
                del cls[rid]
        t_sched, t_grow, n_sched = 0.0, 0.0, 0
        per_it = []
        for it in range(args.iterations):
            ids = np.array(sorted(cls), dtype=np.int32)
            q = np.zeros(len(ids), dtype=SCHED_DTYPE)
            q["id"] = ids
            q["n_new"] = 1
            info = np.array([mgr.query(int(r)) for r in ids], dtype=np.int64).reshape(-1, 3)
            q["ctx_after"] = info[:, 0] + 1
            is_rt = np.array([cls[int(r)] == 0 for r in ids])
            q["remaining_us"] = rng.uniform(2e3, 5e4, len(ids))
            q["m_cpu"] = info[:, 2]
            rt, be = q[is_rt], q[~is_rt]
            n_pend = len(rt) // 4
            pending = rt[:n_pend]
            waiting = np.sort(rt[n_pend:], order="remaining_us", kind="stable")   # the queue's own order
            t0 = time.perf_counter()
            if mode == "per_request":
                got_rt, got_be, _ = schedule(mgr, np.concatenate([pending, waiting]), be, args.batch, coef,
                                             per_request=True)
            else:
                got_rt, got_be, _ = schedule_pulled(mgr, pending, waiting, be, args.batch, coef, per_request=True)
            t1 = time.perf_counter()
            run = got_rt + got_be
            if mode == "per_request":
                for rid in run:
                    try:
                        if mgr.query(rid)[2]:
                            mgr.restore(rid)
                        mgr.grow(rid, 1)
                    except Exception:
                        mgr.release(rid)
                        del cls[rid]
            else:
                _, _, status = mgr.grow_batch(run, np.ones(len(run), dtype=np.int32))
                for i in np.flatnonzero(status):   # requests that could not grow
                    mgr.release(run[i])
                    del cls[run[i]]
            t2 = time.perf_counter()
            t_sched += t1 - t0
            t_grow += t2 - t1
            per_it.append(t2 - t0)
            n_sched += len(run)
            if mode == "batched" and it == 0:
                mgr.validate()
        k = args.iterations
        out[mode] = {"scheduled_per_iteration": round(n_sched / k, 1),
                     "schedule_us_per_iteration": round(t_sched / k * 1e6, 1),
                     "block_management_us_per_iteration": round(t_grow / k * 1e6, 1),
                     "total_us_per_iteration": round((t_sched + t_grow) / k * 1e6, 1),
                     # a shared host's hiccups land in single iterations: the median and p90 beside the mean
                     "total_us_p50": round(float(np.percentile(per_it, 50)) * 1e6, 1),
                     "total_us_p90": round(float(np.percentile(per_it, 90)) * 1e6, 1)}
        mgr.close()
    print(json.dumps(out))


if __name__ == "__main__":
    # run the package's copy of this module (its ctypes types are the ones declared to the library)
    from paper_2504_09590_amd.manager import main as _main
    _main()
