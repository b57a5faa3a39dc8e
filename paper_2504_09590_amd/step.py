"""One mixed RT/BE attention step: KV write, prefill chunks, decode.

The paper's executor concatenates the prefill requests of a batch, then the
decode requests, keeps their shapes in a length table and dispatches each half
to its own attention kernel (Sec. 6). MixedStep is that dispatch over the C ABI:
sequences [0, P) of the batch are prefill chunks and [P, S) decode rows. Their
metadata rows are contiguous slices of the batch's tables, so each half gets
plain pointer offsets into the same device arrays.

Order of one step:  bros_kv_write (all S sequences' new tokens)
                    -> bros_attn_prefill_chunk (rows of sequences [0, P))
                    -> bros_attn_decode (sequences [P, S)).
With overlap=True the prefill runs on a second stream after the write, beside
the decode, so the matrix-core bound and the HBM bound halves share the chip.
With prefill_cus=N the two halves also get disjoint compute units: the
prefill runs on a stream limited to the first N compute units, the write and
the decode on a stream limited to the rest (N a multiple of 32).

With fused=True the prefill and the decode run in one launch
(bros_attn_mixed): every workgroup runs one prefill unit, then takes decode
tiles in proportion to the time its unit left it.

With swap_slots=N every step also checkpoints N slots and restores N slots
(Sec. 5.2) through a SwapLane: the gather before the write, the scatter
before the attention, the host copies on copy engines, one stream per
direction, beside it. With swap_serial=True the copies go on the step's own
stream between its kernels instead. The
slots are early positions of decode sequences, which no write of the step
touches, and the restore puts back the bytes they hold, so the step's outputs
do not change; the step then waits for the copies, so its time is about
max(t_exec, t_swap).
"""

from __future__ import annotations

import numpy as np
import torch

from . import bros
from .swap import SwapLane


class MixedStep:
    def __init__(self, batch, dev: bros.DeviceBatch, overlap: bool = False, prefill_cus: int = 0,
                 swap_slots: int = 0, swap_serial: bool = False, fused: bool = False):
        self.batch = batch
        self.dev = dev
        P, S = batch.num_prefill, batch.num_seqs
        self.P, self.S = P, S
        self.dtype_code = bros.BROS_F32 if batch.dtype == "f32" else bros.BROS_BF16
        hq, d = batch.num_q_heads, batch.head_dim
        self.max_ctx_pre = int(batch.ctx_lens[:P].max()) if P else 0
        self.max_ctx_dec = int(batch.ctx_lens[P:].max()) if S > P else 0
        self.max_q_len = int(np.diff(batch.cu_q).max()) if P else 0
        self.out_prefill = torch.empty_like(dev.q_prefill)
        self.out_decode = torch.empty_like(dev.q_decode)
        ws_dec = bros.bros_attn_workspace_size(bros.BROS_WS_DECODE, self.dtype_code, S - P, hq, d, self.max_ctx_dec)
        ws_pre = bros.bros_attn_workspace_size(bros.BROS_WS_PREFILL, self.dtype_code, int(batch.cu_q[-1]), hq, d,
                                               self.max_ctx_pre) if P else 0
        device = dev.k_pool.device
        self.ws_decode = torch.empty(max(ws_dec, 16), dtype=torch.uint8, device=device) if ws_dec else None
        self.ws_prefill = torch.empty(max(ws_pre, 16), dtype=torch.uint8, device=device) if ws_pre else None
        self.fused = bool(fused)
        if self.fused and (overlap or prefill_cus):
            raise ValueError("the fused launch runs both halves in one grid: no overlap or compute-unit split")
        self.prefill_cus = int(prefill_cus) if P > 0 and S > P else 0
        self.overlap = (overlap or self.prefill_cus > 0) and P > 0 and S > P
        self.main = None   # None: the caller's current stream
        if self.prefill_cus:
            total = torch.cuda.get_device_properties(device).multi_processor_count
            self.side = bros.bros_stream_create_cu_share(0, self.prefill_cus)
            self.main = bros.bros_stream_create_cu_share(self.prefill_cus, total - self.prefill_cus)
        else:
            self.side = torch.cuda.Stream(device=device) if self.overlap else None
        self._ev_written = torch.cuda.Event() if self.overlap else None
        self._ev_prefilled = torch.cuda.Event() if self.overlap else None
        self._ev_enter = torch.cuda.Event()
        self._ev_leave = torch.cuda.Event()
        self.swap = None
        self.swap_serial = bool(swap_serial)
        if swap_slots > 0:
            self._init_swap(int(swap_slots))

    def _init_swap(self, n: int):
        b, d = self.batch, self.dev
        # early positions of the decode sequences, which no write of the step touches
        seqs, pos = [], []
        for depth in range(int(b.ctx_lens.max())):
            for s in range(self.P, self.S):
                if depth < int(b.ctx_lens[s]) - 1 and len(seqs) < n:
                    seqs.append(s)
                    pos.append(depth)
            if len(seqs) >= n:
                break
        if len(seqs) < n:
            raise ValueError(f"the batch's decode sequences hold fewer than {n} untouched slots")
        ids = bros.bros_slot_ids(b.block_tables, b.dir, b.cls, b.num_blocks, seqs, pos)
        bros.bros_check_slot_ids(ids, b.num_blocks)
        self.swap_ids = torch.from_numpy(ids).to(d.k_pool.device)
        hkv, hd = d.k_pool.shape[1], d.k_pool.shape[3]
        self.swap = SwapLane(n, hkv, hd, d.k_pool.dtype, d.k_pool.device, serial=self.swap_serial)
        pin = dict(dtype=d.k_pool.dtype, pin_memory=True)
        # K rows then V rows in one pinned buffer each way: one copy per direction
        self.host_out = torch.empty((2 * n, hkv, hd), **pin)
        self.host_in = torch.empty((2 * n, hkv, hd), **pin)
        self.host_out_k, self.host_out_v = self.host_out[:n], self.host_out[n:]
        self.host_in_k, self.host_in_v = self.host_in[:n], self.host_in[n:]
        # the rows the restore puts back: what the slots hold now
        tk = torch.empty((n, hkv, hd), dtype=d.k_pool.dtype, device=d.k_pool.device)
        tv = torch.empty_like(tk)
        bros.bros_kv_gather(d.k_pool, d.v_pool, self.swap_ids, tk, tv)
        torch.cuda.synchronize()
        self.host_in_k.copy_(tk)
        self.host_in_v.copy_(tv)
        self.swap.prefetch(self.host_in_k, self.host_in_v, n)

    # lazy checkpointing around the write ----------------------------------------
    def swap_out(self, stream):
        self.swap.checkpoint(self.dev.k_pool, self.dev.v_pool, self.swap_ids, self.host_out_k, self.host_out_v,
                             stream)

    def swap_in(self, stream):
        self.swap.restore(self.swap_ids, self.dev.k_pool, self.dev.v_pool, stream)

    def swap_next(self, stream):
        """Prefetch for the next step's restore, then make `stream` wait for
        every copy of this step."""
        self.swap.prefetch(self.host_in_k, self.host_in_v, int(self.swap_ids.numel()), stream=stream)
        self.swap.join(stream)

    def close(self):
        """Releases the compute-unit share streams (after their work is done)."""
        if self.prefill_cus and self.main is not None:
            torch.cuda.synchronize()
            for st in (self.side, self.main):
                bros.bros_stream_destroy(st)
            self.main = self.side = None

    # the three calls --------------------------------------------------------
    def kv_write(self, stream=None):
        d = self.dev
        bros.bros_kv_write(d.k_new, d.v_new, d.k_pool, d.v_pool, d.block_tables, d.dir, d.cls,
                           d.pos0, d.cu_new, stream=stream)

    def prefill(self, stream=None):
        if self.P == 0:
            return
        d, P = self.dev, self.P
        bros.bros_attn_prefill_chunk(self.out_prefill, d.q_prefill, d.cu_q, self.max_q_len, d.k_pool, d.v_pool,
                                     d.block_tables[:P], d.dir[:P], d.cls[:P], d.ctx_lens[:P],
                                     self.max_ctx_pre, workspace=self.ws_prefill, stream=stream)

    def decode(self, stream=None):
        if self.S == self.P:
            return
        d, P = self.dev, self.P
        bros.bros_attn_decode(self.out_decode, d.q_decode, d.k_pool, d.v_pool, d.block_tables[P:], d.dir[P:],
                              d.cls[P:], d.ctx_lens[P:], self.max_ctx_dec, workspace=self.ws_decode,
                              stream=stream)

    def mixed(self, stream=None):
        """Both halves in one launch (bros_attn_mixed)."""
        d, P = self.dev, self.P
        bros.bros_attn_mixed(self.out_prefill, d.q_prefill, d.cu_q, self.max_q_len, self.max_ctx_pre,
                             self.out_decode, d.q_decode, self.max_ctx_dec, d.k_pool, d.v_pool, d.block_tables,
                             d.dir, d.cls, d.ctx_lens, P, workspace=self.ws_decode, stream=stream)

    def run(self, write: bool = True):
        """Enqueue one whole step on the current stream (plus the side stream
        when overlapping); returns (prefill output, decode output)."""
        cur = torch.cuda.current_stream()
        main = self.main if self.main is not None else cur
        if main is not cur:
            self._ev_enter.record(cur)
            main.wait_event(self._ev_enter)
        if self.swap is not None:
            self.swap_out(main)
        if write:
            self.kv_write(main)
        if self.swap is not None:
            self.swap_in(main)
        if self.fused:
            self.mixed(main)
        elif self.overlap:
            self._ev_written.record(main)
            self.side.wait_event(self._ev_written)
            self.prefill(self.side)
            self.decode(main)
            self._ev_prefilled.record(self.side)
            main.wait_event(self._ev_prefilled)
        else:
            self.prefill(main)
            self.decode(main)
        if self.swap is not None:
            self.swap_next(main)
        if main is not cur:
            self._ev_leave.record(main)
            cur.wait_event(self._ev_leave)
        return self.out_prefill, self.out_decode
