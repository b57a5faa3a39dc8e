"""Lazy checkpointing of shared blocks over two copy streams (Sec. 5.2, Sec. 6).

When a write is about to take slots that still hold a peer request's tokens,
only those tokens are saved to CPU memory, and they come back when the peer
is scheduled again. On this device the two halves of that are different kinds
of work. The gather and scatter over scattered 256-byte rows are HBM-bound
and take microseconds (bros_kv_gather / bros_kv_scatter). The host copies are
bound by the host link and run on copy engines (bros_copy_dma), which take no
compute unit from the attention. So a SwapLane gathers into a dense device
staging buffer on the compute stream, copies it to pinned host memory on an
outbound copy stream, copies restored rows into a second staging buffer on an
inbound copy stream ahead of time, and scatters them on the compute stream
before the attention that reads them. The two directions use different copy
engines and run at once: on MI355X a device-to-host and a host-to-device copy
side by side keep about 48 and 57 GB/s. The iteration then costs about
max(t_exec, t_swap), as in the paper's cost model (Sec. 4.1).

Ordering, all on the device (no host synchronisation):
  checkpoint: compute stream  [waits: previous copy-out done] gather -> event
              outbound stream [waits: gather] staging -> pinned host -> event
  prefetch:   inbound stream  [waits: previous scatter done] pinned host -> staging -> event
  restore:    compute stream  [waits: prefetch] scatter -> event
"""

from __future__ import annotations

import numpy as np
import torch

from . import bros


class SwapLane:
    def __init__(self, max_slots: int, num_kv_heads: int, head_dim: int, dtype: torch.dtype, device="cuda",
                 serial: bool = False):
        """serial=True enqueues the host copies on the compute stream itself,
        between the kernels, instead of on copy streams beside them."""
        m = max(int(max_slots), 1)
        self.max_slots = int(max_slots)
        # staging: the n K rows of a call, then its n V rows, so that a host
        # buffer laid out the same way takes both in one copy
        self.staging_out = torch.empty((2 * m, num_kv_heads, head_dim), dtype=dtype, device=device)
        self.staging_in = torch.empty((2 * m, num_kv_heads, head_dim), dtype=dtype, device=device)
        self._row = num_kv_heads * head_dim * self.staging_out.element_size()
        self.serial = bool(serial)
        self.out_stream = None if self.serial else torch.cuda.Stream(device=device)
        self.in_stream = None if self.serial else torch.cuda.Stream(device=device)
        self._gathered = torch.cuda.Event()
        self._copied_out = torch.cuda.Event()
        self._copied_in = torch.cuda.Event()
        self._scattered = torch.cuda.Event()
        self._out_done = torch.cuda.Event()
        self._in_done = torch.cuda.Event()
        self._out_pending = False
        self._in_pending = False
        self._n_in = 0
        # copies requested so far, and how many of them a join already made
        # the compute stream wait for (so that stream needs no second wait)
        self._n_out_copies = self._n_in_copies = 0
        self._joined = (None, 0, 0)
        self.timing = None   # a list to collect ("d2h" | "h2d", start, end) timing events of every copy

    def _mark(self, kind: str, cs):
        if self.timing is None:
            return None
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(cs)
        self.timing.append((kind, a, b))
        return b

    def _close(self, end, cs) -> None:
        if end is not None:
            end.record(cs)

    def _bytes(self, n: int) -> int:
        return n * self._row

    def _span(self, host_k, host_v, n: int):
        """host_k and host_v as one 2n-row view when host_v directly follows
        host_k in the same buffer, else None."""
        if not (host_k.is_contiguous() and host_v.is_contiguous()):
            return None
        if host_k.untyped_storage().data_ptr() != host_v.untyped_storage().data_ptr():
            return None
        if host_v.data_ptr() != host_k.data_ptr() + self._bytes(n):
            return None
        return host_k.as_strided((2 * n,) + tuple(host_k.shape[1:]), host_k.stride())

    def copy_out(self, host_k, host_v, n: int, cs) -> None:
        """The n gathered K and V rows to pinned host memory, on stream cs: one
        copy when host_v follows host_k directly, else two."""
        span = self._span(host_k, host_v, n)
        if span is not None:
            bros.bros_copy_dma(span, self.staging_out, 2 * self._bytes(n), stream=cs)
        else:
            bros.bros_copy_dma(host_k, self.staging_out[:n], self._bytes(n), stream=cs)
            bros.bros_copy_dma(host_v, self.staging_out[n:2 * n], self._bytes(n), stream=cs)

    def copy_in(self, host_k, host_v, n: int, cs) -> None:
        """n K and V rows from pinned host memory into the inbound staging."""
        span = self._span(host_k, host_v, n)
        if span is not None:
            bros.bros_copy_dma(self.staging_in, span, 2 * self._bytes(n), stream=cs)
        else:
            bros.bros_copy_dma(self.staging_in[:n], host_k, self._bytes(n), stream=cs)
            bros.bros_copy_dma(self.staging_in[n:2 * n], host_v, self._bytes(n), stream=cs)

    def _room(self, n: int) -> None:
        if n > self.max_slots:
            raise ValueError(f"{n} slots exceed the lane's {self.max_slots}")

    def checkpoint(self, k_pool, v_pool, slot_ids, host_k, host_v, stream) -> None:
        """Saves the rows at slot_ids (device int32) to host_k/host_v (pinned,
        [>= n][Hkv][D]). Enqueue it before the write that overwrites them."""
        n = int(slot_ids.numel())
        self._room(n)
        if self._out_pending and not self._covered(stream, out=True):
            stream.wait_event(self._copied_out)        # the staging buffer is being copied out
        bros.bros_kv_gather(k_pool, v_pool, slot_ids, self.staging_out[:n], self.staging_out[n:2 * n], num_slots=n,
                            stream=stream)
        self._gathered.record(stream)
        cs = stream if self.serial else self.out_stream
        cs.wait_event(self._gathered)
        t = self._mark("d2h", cs)
        self.copy_out(host_k, host_v, n, cs)
        self._n_out_copies += 1
        self._copied_out.record(cs)
        self._close(t, cs)
        self._out_pending = True

    def prefetch(self, host_k, host_v, n: int, stream=None) -> None:
        """Starts copying n checkpointed rows back to the device (on `stream`
        in serial mode, else on the inbound copy stream)."""
        self._room(n)
        cs = self.in_stream
        if self.serial:
            cs = stream if stream is not None else torch.cuda.current_stream()
        if self._in_pending:
            cs.wait_event(self._scattered)             # the previous restore still reads the buffer
        t = self._mark("h2d", cs)
        self.copy_in(host_k, host_v, n, cs)
        self._n_in_copies += 1
        self._copied_in.record(cs)
        self._close(t, cs)
        self._n_in = n

    def restore(self, slot_ids, k_pool, v_pool, stream) -> None:
        """Scatters the prefetched rows to slot_ids (device int32, as many as
        were prefetched). Enqueue it before the attention that reads them."""
        n = int(slot_ids.numel())
        if n != self._n_in:
            raise ValueError(f"restore of {n} slots after a prefetch of {self._n_in}")
        if not self._covered(stream, out=False):
            stream.wait_event(self._copied_in)
        bros.bros_kv_scatter(self.staging_in[:n], self.staging_in[n:2 * n], slot_ids, k_pool, v_pool, num_slots=n,
                             stream=stream)
        self._scattered.record(stream)
        self._in_pending = True

    def _covered(self, stream, out: bool) -> bool:
        """Whether a join on `stream` already waited for the latest copy of
        that direction."""
        s, n_out, n_in = self._joined
        if self.serial or s is None or s != stream:
            return False
        return n_out == self._n_out_copies if out else n_in == self._n_in_copies

    def join(self, stream) -> None:
        """Makes `stream` wait for every copy enqueued so far."""
        if self.serial:
            return
        self._out_done.record(self.out_stream)
        self._in_done.record(self.in_stream)
        stream.wait_event(self._out_done)
        stream.wait_event(self._in_done)
        self._joined = (stream, self._n_out_copies, self._n_in_copies)


class PlanExecutor:
    """Carries out a block manager's plan (paper_2504_09590_amd.manager) on the
    device, on one stream, in the order the plan requires: the victims are
    gathered and copied to pinned host memory, relocated entries are moved
    (gather into staging, scatter to their new slots), and checkpointed rows
    come back (host to staging, scatter). The step's kv_write follows. Rows
    are kept on the host per (request, position) until restored."""

    def __init__(self, k_pool, v_pool, max_rows: int):
        import torch
        hkv, d = k_pool.shape[1], k_pool.shape[3]
        self.k_pool, self.v_pool = k_pool, v_pool
        self.max_rows = int(max_rows)
        shape = (self.max_rows, hkv, d)
        self.sk = torch.empty(shape, dtype=k_pool.dtype, device=k_pool.device)
        self.sv = torch.empty(shape, dtype=k_pool.dtype, device=k_pool.device)
        self.hk = torch.empty(shape, dtype=k_pool.dtype, pin_memory=True)
        self.hv = torch.empty(shape, dtype=k_pool.dtype, pin_memory=True)
        self.store = {}        # (request, position) -> (K row, V row) on the host
        self._row = self.sk[0].numel() * self.sk.element_size()

    def _ids(self, ids):
        import torch
        return torch.from_numpy(np.ascontiguousarray(ids, dtype=np.int32)).to(self.k_pool.device)

    def execute(self, req: int, plan, stream=None) -> None:
        import torch
        stream = stream if stream is not None else torch.cuda.current_stream()
        for lo in range(0, len(plan.victims), self.max_rows):
            part = plan.victims[lo:lo + self.max_rows]
            n = len(part)
            ids = self._ids(part[:, 2] * 16 + part[:, 3])
            bros.bros_kv_gather(self.k_pool, self.v_pool, ids, self.sk, self.sv, num_slots=n, stream=stream)
            bros.bros_copy_dma(self.hk, self.sk, n * self._row, stream=stream)
            bros.bros_copy_dma(self.hv, self.sv, n * self._row, stream=stream)
            stream.synchronize()
            for i, (r, p, _, _) in enumerate(part):
                self.store[(int(r), int(p))] = (self.hk[i].clone(), self.hv[i].clone())
        for lo in range(0, len(plan.move_src), self.max_rows):
            src, dst = plan.move_src[lo:lo + self.max_rows], plan.move_dst[lo:lo + self.max_rows]
            bros.bros_kv_gather(self.k_pool, self.v_pool, self._ids(src), self.sk, self.sv, num_slots=len(src),
                                stream=stream)
            bros.bros_kv_scatter(self.sk, self.sv, self._ids(dst), self.k_pool, self.v_pool, num_slots=len(dst),
                                 stream=stream)
        for lo in range(0, len(plan.restore_pos), self.max_rows):
            pos, dst = plan.restore_pos[lo:lo + self.max_rows], plan.restore_dst[lo:lo + self.max_rows]
            stream.synchronize()                      # the host rows are reused below
            for i, p in enumerate(pos):
                k, v = self.store.pop((int(req), int(p)))
                self.hk[i].copy_(k)
                self.hv[i].copy_(v)
            n = len(pos)
            bros.bros_copy_dma(self.sk, self.hk, n * self._row, stream=stream)
            bros.bros_copy_dma(self.sv, self.hv, n * self._row, stream=stream)
            bros.bros_kv_scatter(self.sk, self.sv, self._ids(dst), self.k_pool, self.v_pool, num_slots=n,
                                 stream=stream)

    def drop(self, req: int) -> None:
        for key in [k for k in self.store if k[0] == req]:
            del self.store[key]
