"""ctypes binding of libbros_attn.so (declared in include/bros_attn.h).

Argument marshalling only: every step of the paged-attention path runs in the
HIP kernels behind the C ABI. PyTorch supplies device memory and streams.
Functions keep the C names; shapes are read from the tensors. Importing this
module fails loudly when the library has not been built: there is no fallback.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libbros_attn.so")

BROS_F32, BROS_BF16 = 0, 1
BROS_RT, BROS_BE = 0, 1
BROS_WS_DECODE, BROS_WS_PREFILL = 0, 1
STATUS = {0: "BROS_OK", -1: "BROS_E_NULL", -2: "BROS_E_SHAPE", -3: "BROS_E_DTYPE",
          -4: "BROS_E_UNSUPPORTED", -5: "BROS_E_WORKSPACE", -6: "BROS_E_HIP", -7: "BROS_E_TABLE",
          -8: "BROS_E_NOMEM"}

EXPORTED = ["bros_status_str", "bros_last_error", "bros_abi_version", "bros_kv_write",
            "bros_attn_decode", "bros_attn_decode_noalloc", "bros_attn_prefill_chunk", "bros_attn_mixed", "bros_attn_workspace_size",
            "bros_check_batch", "bros_stream_create_cu_share", "bros_stream_destroy",
            "bros_kv_gather", "bros_kv_scatter", "bros_check_slot_ids", "bros_copy_dma", "bros_slot_ids",
            "bros_mgr_create", "bros_mgr_destroy", "bros_mgr_add_request", "bros_mgr_release", "bros_mgr_grow",
            "bros_mgr_restore", "bros_mgr_query", "bros_mgr_table", "bros_mgr_free_blocks", "bros_mgr_validate", "bros_mgr_available",
            "bros_mgr_entries_needed", "bros_mgr_preemption_table", "bros_schedule", "bros_next_batch_size",
            "bros_mgr_grow_batch", "bros_mgr_plan_bound", "bros_schedule_pulled", "bros_set_decode_kernel_events"]


class BrosError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2504_09590_amd.build`")
    # Load torch's HIP runtime first: the library's libamdhip64.so.7 dependency
    # then resolves to that already-mapped copy, so the process runs ONE HIP
    # runtime and device pointers and streams from torch are valid here.
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    P, I, F, Z = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
    lib.bros_status_str.argtypes = [ctypes.c_int]
    lib.bros_status_str.restype = ctypes.c_char_p
    lib.bros_last_error.argtypes = []
    lib.bros_last_error.restype = ctypes.c_char_p
    lib.bros_abi_version.argtypes = []
    lib.bros_abi_version.restype = ctypes.c_int
    lib.bros_kv_write.argtypes = [P, P, I, P, P, I, P, I, P, P, I, P, P, I, I, I, I, I, P]
    lib.bros_kv_write.restype = ctypes.c_int
    lib.bros_attn_decode.argtypes = [P, P, P, P, I, P, I, P, P, I, P, I, I, I, I, I, I, F, I, P, Z, P]
    lib.bros_attn_decode.restype = ctypes.c_int
    lib.bros_attn_decode_noalloc.argtypes = [P, P, P, P, I, P, I, P, P, I, P, I, I, I, I, I, I, F, I, P]
    lib.bros_attn_decode_noalloc.restype = ctypes.c_int
    lib.bros_attn_prefill_chunk.argtypes = [P, P, P, I, I, P, P, I, P, I, P, P, I, P, I, I, I, I, I, I, F, I, P, Z, P]
    lib.bros_attn_prefill_chunk.restype = ctypes.c_int
    lib.bros_attn_mixed.argtypes = [P, P, P, I, I, I, I, P, P, I, I, P, P, I, P, I, P, P, I, P, I, I, I, I, F, I, P, Z, P]
    lib.bros_attn_mixed.restype = ctypes.c_int
    lib.bros_set_decode_kernel_events.argtypes = [P, P]
    lib.bros_set_decode_kernel_events.restype = ctypes.c_int
    lib.bros_attn_workspace_size.argtypes = [I, I, I, I, I, I]
    lib.bros_attn_workspace_size.restype = Z
    lib.bros_check_batch.argtypes = [P, I, P, P, I, P, I, I, I, I]
    lib.bros_check_batch.restype = ctypes.c_int
    lib.bros_stream_create_cu_share.argtypes = [I, I, ctypes.POINTER(ctypes.c_void_p)]
    lib.bros_stream_create_cu_share.restype = ctypes.c_int
    lib.bros_stream_destroy.argtypes = [P]
    lib.bros_stream_destroy.restype = ctypes.c_int
    lib.bros_kv_gather.argtypes = [P, P, I, P, I, P, P, I, I, I, I, P]
    lib.bros_kv_gather.restype = ctypes.c_int
    lib.bros_kv_scatter.argtypes = [P, P, P, I, P, P, I, I, I, I, I, P]
    lib.bros_kv_scatter.restype = ctypes.c_int
    lib.bros_check_slot_ids.argtypes = [P, I, I]
    lib.bros_check_slot_ids.restype = ctypes.c_int
    lib.bros_slot_ids.argtypes = [P, I, P, P, I, I, I, P, P, I, P]
    lib.bros_slot_ids.restype = ctypes.c_int
    lib.bros_copy_dma.argtypes = [P, P, Z, P]
    lib.bros_copy_dma.restype = ctypes.c_int
    from . import manager as _m   # host block manager and scheduler signatures
    _m.declare(lib)
    return lib


LIB = _load()


def _check(status: int) -> None:
    if status != 0:
        raise BrosError(status, LIB.bros_last_error().decode())


def _ptr(t) -> int | None:
    """Device (or host numpy) address of a contiguous buffer; None passes NULL."""
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        if not t.flags["C_CONTIGUOUS"]:
            raise ValueError("numpy array must be C-contiguous")
        return t.ctypes.data
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return BROS_F32
    if t.dtype == torch.bfloat16:
        return BROS_BF16
    raise ValueError(f"unsupported dtype {t.dtype}")


def _stream(stream) -> int | None:
    if stream is not None:
        return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
    import torch
    return torch.cuda.current_stream().cuda_stream


def _numel0(t) -> int:
    return 0 if t is None else int(t.shape[0])


def _dir_mode(dir, block_tables) -> int:
    """0 for one flag per sequence, 1 for the direction table (one flag per
    block-table entry, shaped like the tables)."""
    if dir is None or len(dir.shape) == 1:
        return 0
    if tuple(dir.shape) != tuple(block_tables.shape):
        raise ValueError(f"direction table {tuple(dir.shape)} must match block tables {tuple(block_tables.shape)}")
    return 1


def bros_kv_write(k_new, v_new, k_pool, v_pool, block_tables, dir, cls, pos0, cu_new, stream=None):
    """Store new tokens' K/V ([Tn][Hkv][D]) in their bidirectional slots of the pools."""
    nb, hkv, bs, d = (int(x) for x in k_pool.shape)
    _check(LIB.bros_kv_write(_ptr(k_new), _ptr(v_new), _numel0(k_new), _ptr(k_pool), _ptr(v_pool), nb,
                             _ptr(block_tables), int(block_tables.shape[1]), _ptr(dir), _ptr(cls),
                             _dir_mode(dir, block_tables), _ptr(pos0), _ptr(cu_new), int(cu_new.shape[0]) - 1, hkv, d, bs,
                             _dtype_code(k_pool), _stream(stream)))


def bros_set_decode_kernel_events(before=None, after=None):
    """Measurement hook: later bf16 decode calls record these torch.cuda.Events
    (timing enabled, each recorded once already so that it exists) right
    before and right after their decode kernel; None, None turns it off."""
    handle = (lambda e: None if e is None else ctypes.c_void_p(e.cuda_event))
    _check(LIB.bros_set_decode_kernel_events(handle(before), handle(after)))


def bros_attn_workspace_size(kind: int, dtype: int, num_rows: int, num_q_heads: int,
                             head_dim: int, max_ctx: int) -> int:
    return int(LIB.bros_attn_workspace_size(kind, dtype, num_rows, num_q_heads, head_dim, max_ctx))


def bros_attn_decode(out, q, k_pool, v_pool, block_tables, dir, cls, ctx_lens, max_ctx: int,
                     scale: float = 0.0, workspace=None, stream=None):
    """out[s][h] = attention of q[s][h] over sequence s's paged context."""
    nb, hkv, bs, d = (int(x) for x in k_pool.shape)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(LIB.bros_attn_decode(_ptr(out), _ptr(q), _ptr(k_pool), _ptr(v_pool), nb, _ptr(block_tables),
                                int(block_tables.shape[1]), _ptr(dir), _ptr(cls), _dir_mode(dir, block_tables),
                                _ptr(ctx_lens), int(max_ctx), int(ctx_lens.shape[0]), int(q.shape[1]), hkv, d, bs,
                                float(scale), _dtype_code(q), _ptr(workspace), ws_bytes, _stream(stream)))


def bros_attn_decode_noalloc(out, q, k_pool, v_pool, block_tables, dir, cls, ctx_lens, max_ctx: int,
                             scale: float = 0.0, stream=None):
    """bros_attn_decode with the library's static scratch array as its workspace
    (for callers that cannot allocate); rejects batches beyond the array."""
    nb, hkv, bs, d = (int(x) for x in k_pool.shape)
    _check(LIB.bros_attn_decode_noalloc(_ptr(out), _ptr(q), _ptr(k_pool), _ptr(v_pool), nb, _ptr(block_tables),
                                        int(block_tables.shape[1]), _ptr(dir), _ptr(cls),
                                        _dir_mode(dir, block_tables), _ptr(ctx_lens), int(max_ctx),
                                        int(ctx_lens.shape[0]), int(q.shape[1]), hkv, d, bs, float(scale),
                                        _dtype_code(q), _stream(stream)))


def bros_attn_prefill_chunk(out, q, cu_q, max_q_len: int, k_pool, v_pool, block_tables, dir, cls,
                            ctx_lens, max_ctx: int, scale: float = 0.0, workspace=None, stream=None):
    """Causal attention of each prefill chunk's rows over its sequence's paged context."""
    nb, hkv, bs, d = (int(x) for x in k_pool.shape)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(LIB.bros_attn_prefill_chunk(_ptr(out), _ptr(q), _ptr(cu_q), int(q.shape[0]), int(max_q_len),
                                       _ptr(k_pool), _ptr(v_pool), nb, _ptr(block_tables),
                                       int(block_tables.shape[1]), _ptr(dir), _ptr(cls),
                                       _dir_mode(dir, block_tables), _ptr(ctx_lens), int(max_ctx), int(ctx_lens.shape[0]), int(q.shape[1]), hkv, d, bs,
                                       float(scale), _dtype_code(q), _ptr(workspace), ws_bytes,
                                       _stream(stream)))


def bros_attn_mixed(out_prefill, q_prefill, cu_q, max_q_len: int, max_ctx_prefill: int, out_decode, q_decode,
                    max_ctx_decode: int, k_pool, v_pool, block_tables, dir, cls, ctx_lens, num_prefill_seqs: int,
                    scale: float = 0.0, workspace=None, stream=None):
    """Prefill chunks (metadata rows [0, P)) and decode rows (rows [P, S)) of
    one concatenated batch in one launch."""
    nb, hkv, bs, d = (int(x) for x in k_pool.shape)
    P = int(num_prefill_seqs)
    D = int(ctx_lens.shape[0]) - P
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    qp = q_prefill if q_prefill is not None and q_prefill.numel() else None
    _check(LIB.bros_attn_mixed(_ptr(out_prefill) if qp is not None else None, _ptr(qp), _ptr(cu_q),
                               0 if qp is None else int(qp.shape[0]), int(max_q_len), P, int(max_ctx_prefill),
                               _ptr(out_decode) if D else None, _ptr(q_decode) if D else None, D, int(max_ctx_decode),
                               _ptr(k_pool), _ptr(v_pool), nb, _ptr(block_tables), int(block_tables.shape[1]),
                               _ptr(dir), _ptr(cls), _dir_mode(dir, block_tables), _ptr(ctx_lens),
                               int((q_decode if D else q_prefill).shape[1]), hkv, d, bs, float(scale),
                               _dtype_code(k_pool), _ptr(workspace), ws_bytes, _stream(stream)))


def bros_check_batch(block_tables: np.ndarray, dir, cls, ctx_lens: np.ndarray, num_blocks: int,
                     check_slot_disjointness: bool = True, block_size: int = 16) -> None:
    """Host-side consistency check; raises BrosError naming the first problem."""
    bt = np.ascontiguousarray(block_tables, dtype=np.int32)
    cl = np.ascontiguousarray(ctx_lens, dtype=np.int32)
    dr = None if dir is None else np.ascontiguousarray(dir, dtype=np.int8)
    cs = None if cls is None else np.ascontiguousarray(cls, dtype=np.uint8)
    _check(LIB.bros_check_batch(_ptr(bt), int(bt.shape[1]) if bt.ndim == 2 else 0, _ptr(dr), _ptr(cs),
                                _dir_mode(dr, bt), _ptr(cl), int(cl.shape[0]), int(num_blocks), int(block_size),
                                1 if check_slot_disjointness else 0))


def bros_kv_gather(k_pool, v_pool, slot_ids, k_out, v_out, num_slots: int | None = None, stream=None):
    """Rows of the pools at slot ids (block * 16 + slot) into dense [n][Hkv][D]
    buffers (device memory, or pinned host memory). n defaults to len(slot_ids)."""
    n = _numel0(slot_ids) if num_slots is None else int(num_slots)
    nb, hkv, _, d = k_pool.shape
    _check(LIB.bros_kv_gather(_ptr(k_pool), _ptr(v_pool), int(nb), _ptr(slot_ids), n, _ptr(k_out), _ptr(v_out),
                              int(hkv), int(d), 16, _dtype_code(k_pool), _stream(stream)))


def bros_kv_scatter(k_in, v_in, slot_ids, k_pool, v_pool, num_slots: int | None = None, stream=None):
    """Dense [n][Hkv][D] rows back into the pools at slot ids; ids outside the
    pool are skipped."""
    n = _numel0(slot_ids) if num_slots is None else int(num_slots)
    nb, hkv, _, d = k_pool.shape
    _check(LIB.bros_kv_scatter(_ptr(k_in), _ptr(v_in), _ptr(slot_ids), n, _ptr(k_pool), _ptr(v_pool), int(nb),
                               int(hkv), int(d), 16, _dtype_code(k_pool), _stream(stream)))


def bros_copy_dma(dst, src, nbytes: int | None = None, stream=None) -> None:
    """Asynchronous copy on a DMA engine between device and/or pinned host
    tensors (contiguous); nbytes defaults to the size of src."""
    n = src.numel() * src.element_size() if nbytes is None else int(nbytes)
    if n > dst.numel() * dst.element_size() or n > src.numel() * src.element_size():
        raise ValueError("copy larger than a buffer")
    _check(LIB.bros_copy_dma(_ptr(dst), _ptr(src), n, _stream(stream)))


def bros_slot_ids(block_tables: np.ndarray, dir, cls, num_blocks: int, seqs, positions) -> np.ndarray:
    """Host: slot ids (block * 16 + slot) of (sequence, position) pairs under
    the batch's tables and directions; raises BrosError naming a bad pair."""
    bt = np.ascontiguousarray(block_tables, dtype=np.int32)
    dr = None if dir is None else np.ascontiguousarray(dir, dtype=np.int8)
    cs = None if cls is None else np.ascontiguousarray(cls, dtype=np.uint8)
    sq = np.ascontiguousarray(seqs, dtype=np.int32)
    ps = np.ascontiguousarray(positions, dtype=np.int32)
    if sq.shape != ps.shape:
        raise ValueError("seqs and positions must have the same length")
    out = np.empty(sq.shape[0], dtype=np.int32)
    _check(LIB.bros_slot_ids(_ptr(bt), int(bt.shape[1]), _ptr(dr), _ptr(cs), _dir_mode(dr, bt), int(bt.shape[0]),
                             int(num_blocks), _ptr(sq), _ptr(ps), int(sq.shape[0]), _ptr(out)))
    return out


def bros_check_slot_ids(slot_ids: np.ndarray, num_blocks: int) -> None:
    """Host check that the ids inside the pool are distinct; raises BrosError."""
    ids = np.ascontiguousarray(slot_ids, dtype=np.int32)
    _check(LIB.bros_check_slot_ids(_ptr(ids), int(ids.shape[0]), int(num_blocks)))


def bros_stream_create_cu_share(first_cu: int, num_cus: int):
    """A torch stream wrapping a new hipStream_t limited to compute units
    [first_cu, first_cu + num_cus); release it with bros_stream_destroy."""
    import torch
    handle = ctypes.c_void_p()
    _check(LIB.bros_stream_create_cu_share(int(first_cu), int(num_cus), ctypes.byref(handle)))
    return torch.cuda.ExternalStream(handle.value)


def bros_stream_destroy(stream) -> None:
    _check(LIB.bros_stream_destroy(ctypes.c_void_p(_stream(stream))))


# ---------------------------------------------------------------------------
# device copies of a generated batch (marshalling for tests and the benchmark)
# ---------------------------------------------------------------------------

@dataclass
class DeviceBatch:
    k_pool: object
    v_pool: object
    block_tables: object
    dir: object
    cls: object
    ctx_lens: object
    cu_q: object
    q_prefill: object
    q_decode: object
    cu_new: object
    pos0: object
    k_new: object
    v_new: object


def _tensor(x: np.ndarray, dtype: str | None, device):
    import torch
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(x))
    return t.to(device)


def to_device(batch, device="cuda") -> DeviceBatch:
    """Copy a workload.Batch to device tensors (bf16 bit patterns become bfloat16)."""
    dt = batch.dtype
    return DeviceBatch(
        k_pool=_tensor(batch.k_pool, dt, device), v_pool=_tensor(batch.v_pool, dt, device),
        block_tables=_tensor(batch.block_tables, None, device), dir=_tensor(batch.dir, None, device),
        cls=_tensor(batch.cls, None, device), ctx_lens=_tensor(batch.ctx_lens, None, device),
        cu_q=_tensor(batch.cu_q, None, device), q_prefill=_tensor(batch.q_prefill, dt, device),
        q_decode=_tensor(batch.q_decode, dt, device), cu_new=_tensor(batch.cu_new, None, device),
        pos0=_tensor(batch.pos0, None, device), k_new=_tensor(batch.k_new, dt, device),
        v_new=_tensor(batch.v_new, dt, device))


def to_host_bits(t) -> np.ndarray:
    """Device tensor -> numpy (bf16 as uint16 bit patterns, fp32 as float32)."""
    import torch
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()
