/*
 * bros_attn.h -- C ABI of the MI355X (gfx950) bidirectional paged-attention step.
 *
 * One serving iteration over a mixed batch of real-time (RT) and best-effort
 * (BE) requests whose KV cache lives in ONE shared pool of 16-slot blocks with
 * the bidirectional layout of "Efficient LLM Serving on Hybrid Real-time and
 * Best-effort Requests" (arXiv 2504.09590):
 *
 *   - Sec. 5.1 (Block Structure): a block can hold one RT and one BE request;
 *     the RT request's tokens fill its slots from the left end, the BE
 *     request's from the right end; a request may span several blocks.
 *   - Sec. 5.2 (Block Management, lazy checkpointing): while free slots remain
 *     each request treats a shared block as its own, so entry i of a request's
 *     block table holds its logical positions [16 i, 16 i + 16).
 *   - Sec. 6 (Implementation): the attention kernel receives the block tables
 *     plus a direction flag telling whether a block's slots are walked from the
 *     left or from the right; prefill rows of the batch are concatenated along
 *     the token axis with a length table, decode rows follow.
 *
 * Slot of logical position p of a sequence with direction d:
 *     block = block_tables[s][p / 16],  slot = (d == +1) ? p % 16 : 15 - p % 16.
 *
 * COMMON CONVENTIONS
 *   Pointers named *_pool, q, out, k_new, v_new, block_tables, dir, cls,
 *   ctx_lens, pos0, cu_new, cu_q and workspace are HIP DEVICE pointers, owned
 *   by the caller, row-major and contiguous. The library allocates nothing per
 *   call, keeps no state between calls, never synchronizes, and enqueues its
 *   kernels on `stream` (a hipStream_t; NULL = the null stream). Calls on
 *   different streams touching disjoint outputs may run concurrently.
 *
 *   Pool layout:  k_pool, v_pool  [num_blocks][num_kv_heads][16][head_dim]
 *                 (one (block, KV head) tile = 16 x head_dim contiguous values).
 *   dtype:        BROS_F32 or BROS_BF16; q, pools, k_new/v_new and out share it.
 *                 Arithmetic accumulates in fp32; bf16 outputs are rounded to
 *                 nearest-even.
 *   dir:          int8 [num_seqs], +1 (left-to-right) or -1 (right-to-left).
 *                 May be NULL: then the direction is derived from cls
 *                 (RT -> +1, BE -> -1), which is the layout of Sec. 5.1.
 *   dir_per_entry: 0 for the form above; 1 when dir is the paper's
 *                 direction table (Sec. 6), int8 [num_seqs][max_blocks_per_seq]
 *                 with one flag per block-table entry: positions of entry i
 *                 are walked in that entry's direction. Requires dir.
 *   cls:          uint8 [num_seqs], BROS_RT or BROS_BE. Only consulted when
 *                 dir is NULL; it has no other numerical effect. May be NULL
 *                 when dir is given.
 *   block_tables: int32 [num_seqs][max_blocks_per_seq]; entries at index
 *                 >= ceil(ctx / 16) are never read.
 *   ctx_lens:     int32 [num_seqs], tokens in the cache AFTER this step's
 *                 writes (a decode sequence's count includes its new token).
 *   Supported shapes: block_size == 16, head_dim == 128, num_q_heads a
 *   multiple of num_kv_heads with group size 1, 2, 4 or 8.
 *
 *   Block-table contents are NOT validated in the hot path (that would need a
 *   device-to-host copy). The kernels never touch memory outside the buffers
 *   whatever the tables hold: an entry outside [0, num_blocks) or a context
 *   longer than max_blocks_per_seq * 16 makes the affected tokens contribute
 *   nothing (attention) or not be written (kv_write). bros_check_batch() runs
 *   the full consistency check on host copies.
 *
 * ERRORS
 *   Every entry point returns BROS_OK (0) or a negative status; nothing is
 *   launched when the status is negative, except BROS_E_HIP which reports a
 *   launch failure. bros_last_error() returns a thread-local message describing
 *   the most recent failure on the calling thread. No exception crosses the ABI.
 */
#ifndef BROS_ATTN_H
#define BROS_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum bros_dtype { BROS_F32 = 0, BROS_BF16 = 1 };
enum bros_class { BROS_RT = 0, BROS_BE = 1 };
enum bros_status {
  BROS_OK = 0,
  BROS_E_NULL = -1,        /* a required pointer is NULL                               */
  BROS_E_SHAPE = -2,       /* inconsistent sizes (Hq % Hkv, negative counts, ...)        */
  BROS_E_DTYPE = -3,       /* dtype is neither BROS_F32 nor BROS_BF16                   */
  BROS_E_UNSUPPORTED = -4, /* block_size != 16, head_dim != 128, group not in {1,2,4,8} */
  BROS_E_WORKSPACE = -5,   /* workspace missing or smaller than the size query's answer */
  BROS_E_HIP = -6,         /* a HIP launch failed; message carries hipGetErrorString    */
  BROS_E_TABLE = -7,       /* bros_check_batch found an inconsistent batch               */
  BROS_E_NOMEM = -8        /* the block manager found no block for a request            */
};
enum bros_workspace_kind { BROS_WS_DECODE = 0, BROS_WS_PREFILL = 1 };

/* Static string naming a status code. */
const char* bros_status_str(int status);
/* Message of the last failure on the calling thread ("" if none). */
const char* bros_last_error(void);
/* ABI version of this library (increments on any signature change). */
int bros_abi_version(void);

/*
 * bros_kv_write -- store this step's new tokens in their bidirectional slots.
 *
 * Defines: Sec. 5.1 (RT fills a block from the left, BE from the right) with
 * the exclusive view of Sec. 5.2. For every sequence s and every new token t
 * in [cu_new[s], cu_new[s+1]), at logical position p = pos0[s] + t - cu_new[s]:
 *     k_pool[block][h][slot][:] = k_new[t][h][:]   for every KV head h,
 *     v_pool[block][h][slot][:] = v_new[t][h][:],
 * with (block, slot) from the mapping above. Pure data movement: the pool
 * bytes at every written slot equal the source bytes; no other byte changes.
 * Two sequences sharing a block write disjoint slots in the same launch.
 *
 *   k_new, v_new : [num_new_tokens][num_kv_heads][head_dim]
 *   pos0         : int32 [num_seqs], logical position of each sequence's first new token
 *   cu_new       : int32 [num_seqs + 1], prefix offsets of new tokens; cu_new[0] = 0,
 *                  cu_new[num_seqs] = num_new_tokens
 * num_new_tokens == 0 is a no-op. A token whose block-table entry is out of
 * range (see COMMON CONVENTIONS) is skipped. num_kv_heads above 16384 is
 * BROS_E_UNSUPPORTED.
 */
int bros_kv_write(const void* k_new, const void* v_new, int32_t num_new_tokens,
                  void* k_pool, void* v_pool, int32_t num_blocks,
                  const int32_t* block_tables, int32_t max_blocks_per_seq,
                  const int8_t* dir, const uint8_t* cls, int32_t dir_per_entry,
                  const int32_t* pos0, const int32_t* cu_new,
                  int32_t num_seqs, int32_t num_kv_heads, int32_t head_dim,
                  int32_t block_size, int32_t dtype, void* stream);

/*
 * bros_attn_decode -- one query row per sequence over its whole paged context.
 *
 * Defines: the decode attention of Sec. 2.1 (the new token attends to the
 * cached keys/values of all earlier tokens and itself) run over the
 * direction-aware paged layout of Sec. 5.1 / Sec. 6. For sequence s and query
 * head h, with g = h / (num_q_heads / num_kv_heads) and the keys/values of
 * positions p < ctx_lens[s] gathered through the block table:
 *     out[s][h][:] = sum_p softmax_p(scale * q[s][h] . K[p][g]) * V[p][g][:].
 * A sequence with ctx_lens[s] <= 0 gets a zero output row.
 *
 *   q, out       : [num_seqs][num_q_heads][head_dim]
 *   max_ctx      : host-side upper bound of every ctx_lens[s]; sizes the grid
 *                  and the workspace without a device-to-host copy. Contexts
 *                  above it are truncated to max_ctx.
 *   scale        : softmax scale; <= 0 selects 1 / sqrt(head_dim)
 *   workspace    : device scratch of at least
 *                  bros_attn_workspace_size(BROS_WS_DECODE, dtype, num_seqs,
 *                  num_q_heads, head_dim, max_ctx) bytes, 16-byte aligned (may
 *                  be NULL when that size is 0); overwritten by every call.
 *                  bf16: the first tile of each row and the partial results
 *                  of (row, KV head) contexts shared by several workers (the
 *                  grid's waves each take an equal share of the 16-slot
 *                  tiles); its size does not depend on max_ctx. fp32: split-K
 *                  partials, needed only when a context spans several splits.
 *                  Two calls that share a workspace must not overlap in time.
 * Errors: BROS_E_SHAPE also when bf16 num_seqs * num_kv_heads *
 * ceil(max_ctx / 16) exceeds 2^31 - 1.
 */
int bros_attn_decode(void* out, const void* q,
                     const void* k_pool, const void* v_pool, int32_t num_blocks,
                     const int32_t* block_tables, int32_t max_blocks_per_seq,
                     const int8_t* dir, const uint8_t* cls, int32_t dir_per_entry, const int32_t* ctx_lens,
                     int32_t max_ctx, int32_t num_seqs, int32_t num_q_heads,
                     int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                     float scale, int32_t dtype, void* workspace, size_t workspace_bytes,
                     void* stream);

/*
 * bros_attn_prefill_chunk -- causal attention of RT prefill chunks over the pool.
 *
 * Defines: the prefill half of the mixed batch of Sec. 6 (prefill rows
 * concatenated along the token axis, their shapes in a length table), with
 * chunked prefill on top of already-cached context (Sec. 2.2 / Sec. 8). Rows
 * of sequence s are q[cu_q[s] .. cu_q[s+1]); with n = cu_q[s+1] - cu_q[s] and
 * c0 = ctx_lens[s] - n (the chunk's K/V already stored by bros_kv_write), row j
 * sits at position c0 + j and attends to positions 0 .. c0 + j (diagonal
 * inclusive), with the same head grouping and gather as bros_attn_decode.
 * Sequences with n == 0 are skipped.
 *
 *   q, out       : [num_q_tokens][num_q_heads][head_dim]
 *   cu_q         : int32 [num_seqs + 1], prefix offsets; cu_q[num_seqs] = num_q_tokens
 *   max_q_len    : host-side upper bound of every n (sizes the grid)
 *   max_ctx      : host-side upper bound of every ctx_lens[s]
 *   workspace    : at least bros_attn_workspace_size(BROS_WS_PREFILL, dtype,
 *                  num_q_tokens, num_q_heads, head_dim, max_ctx) bytes,
 *                  16-byte aligned; owned by the caller, contents undefined
 *                  after the call.
 * bf16 runs the QK^T and PV products on the matrix cores (P is rounded to bf16
 * before PV) for max_ctx <= 32768. There the workspace is optional (NULL, or
 * one smaller than the query, is accepted): with it, when the call's (row
 * tile, KV head) units are fewer than the compute units, long units are split
 * over key ranges whose partial results are merged, so idle compute units
 * take a share; without it every unit runs whole. The merged rows differ from
 * the unsplit ones by rounding only. fp32, and bf16 beyond that context, run
 * a vector-ALU path that requires the workspace (BROS_E_WORKSPACE otherwise).
 */
int bros_attn_prefill_chunk(void* out, const void* q, const int32_t* cu_q,
                            int32_t num_q_tokens, int32_t max_q_len,
                            const void* k_pool, const void* v_pool, int32_t num_blocks,
                            const int32_t* block_tables, int32_t max_blocks_per_seq,
                            const int8_t* dir, const uint8_t* cls, int32_t dir_per_entry, const int32_t* ctx_lens,
                            int32_t max_ctx, int32_t num_seqs, int32_t num_q_heads,
                            int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                            float scale, int32_t dtype, void* workspace, size_t workspace_bytes,
                            void* stream);

/*
 * bros_attn_mixed -- the prefill chunks and the decode rows of one mixed batch
 * in one launch.
 *
 * Defines: the executor's batch of Sec. 6 -- prefill requests concatenated
 * along the token axis with their shapes in a length table, decode requests
 * after them -- computed in a single grid. The metadata rows (block_tables,
 * dir, cls, ctx_lens) hold the prefill sequences first, rows [0,
 * num_prefill_seqs), then the decode sequences, rows [num_prefill_seqs,
 * num_prefill_seqs + num_decode_seqs). The results equal those of
 *   bros_attn_prefill_chunk(out_prefill, q_prefill, cu_q, ... rows [0, P) ...)
 *   bros_attn_decode(out_decode, q_decode, ... rows [P, P + D) ...)
 * up to rounding (the decode's contexts may be cut between workers at other
 * places). Each workgroup first runs one prefill unit and then takes decode
 * tiles in proportion to the time its unit leaves it, so the prefill's
 * uneven units no longer leave compute units idle.
 *
 *   out_prefill, q_prefill : [num_q_tokens][num_q_heads][head_dim]; cu_q [P + 1]
 *   out_decode, q_decode   : [num_decode_seqs][num_q_heads][head_dim]
 *   max_ctx_prefill, max_ctx_decode : host upper bounds of each half's contexts
 *   workspace : at least bros_attn_workspace_size(BROS_WS_DECODE, BROS_BF16,
 *               num_decode_seqs, num_q_heads, head_dim, max_ctx_decode) bytes,
 *               16-byte aligned, as for bros_attn_decode.
 * bf16 only, prefill contexts up to 32768 (BROS_E_UNSUPPORTED otherwise: use
 * the two calls). With no prefill rows it is bros_attn_decode, with no decode
 * rows bros_attn_prefill_chunk; when the prefill has more units than one grid
 * holds (two workgroups per compute unit) it runs the two calls in turn.
 * Errors as for the two calls.
 */
int bros_attn_mixed(void* out_prefill, const void* q_prefill, const int32_t* cu_q, int32_t num_q_tokens,
                    int32_t max_q_len, int32_t num_prefill_seqs, int32_t max_ctx_prefill,
                    void* out_decode, const void* q_decode, int32_t num_decode_seqs, int32_t max_ctx_decode,
                    const void* k_pool, const void* v_pool, int32_t num_blocks,
                    const int32_t* block_tables, int32_t max_blocks_per_seq,
                    const int8_t* dir, const uint8_t* cls, int32_t dir_per_entry, const int32_t* ctx_lens,
                    int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                    float scale, int32_t dtype, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Bytes of device workspace the call `kind` needs for `num_rows` query rows
 * (num_seqs for decode, num_q_tokens for prefill). Pure host arithmetic; it
 * does not know num_kv_heads and sizes bf16 decode for groups of up to 8
 * query heads. For the bf16 prefill on the matrix cores (max_ctx <= 32768)
 * it returns the size of the optional split workspace, the same for every
 * call. Returns 0 for unsupported arguments.
 */
size_t bros_attn_workspace_size(int32_t kind, int32_t dtype, int32_t num_rows,
                                int32_t num_q_heads, int32_t head_dim, int32_t max_ctx);

/*
 * bros_attn_decode_noalloc -- bros_attn_decode without a caller workspace.
 *
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc. Same
 * arguments, meaning and results as bros_attn_decode (the same kernels run),
 * minus the workspace: the call uses a static device array of
 * BROS_NOALLOC_SCRATCH_BYTES bytes that every GPU the library runs on holds
 * until the process ends. It allocates and frees nothing. The caller still
 * owns q, out, the pools and the metadata.
 *
 * Limit: a batch whose bros_attn_workspace_size(BROS_WS_DECODE, ...) exceeds
 * BROS_NOALLOC_SCRATCH_BYTES is rejected with BROS_E_WORKSPACE before
 * anything is launched (bf16: about num_seqs * num_q_heads * 520 bytes plus
 * 17 MiB, so up to about 60 000 (row, query head) pairs).
 * All calls on one GPU share that GPU's array and it keeps the last call's
 * contents: calls that overlap in time on one GPU (two streams, two threads)
 * race on it and must be serialised by the caller. The first call on a device
 * resolves the array's address there (BROS_E_HIP if the runtime cannot).
 */
#define BROS_NOALLOC_SCRATCH_BYTES (48u << 20)
int bros_attn_decode_noalloc(void* out, const void* q,
                             const void* k_pool, const void* v_pool, int32_t num_blocks,
                             const int32_t* block_tables, int32_t max_blocks_per_seq,
                             const int8_t* dir, const uint8_t* cls, int32_t dir_per_entry,
                             const int32_t* ctx_lens, int32_t max_ctx, int32_t num_seqs,
                             int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                             int32_t block_size, float scale, int32_t dtype, void* stream);

/*
 * bros_kv_gather / bros_kv_scatter -- lazy checkpointing of shared blocks.
 *
 * Defines: Sec. 5.2 (lazy checkpointing): once a shared block has no empty
 * slot left, only the tokens of the peer request that a write is about to
 * overwrite are copied to CPU memory, and they are copied back when that
 * request is scheduled again; Sec. 6: dedicated kernels fetch and store KV
 * in non-contiguous GPU memory and separate streams carry the host copies.
 *
 * A slot is named by its id, block * 16 + slot. For i in [0, num_slots) and
 * every KV head h:
 *   gather:   k_out[i][h][:] = k_pool[id_i / 16][h][id_i % 16][:]  (v likewise);
 *             a row whose id lies outside [0, num_blocks * 16) is written as zeros.
 *   scatter:  k_pool[id_i / 16][h][id_i % 16][:] = k_in[i][h][:]    (v likewise);
 *             an id outside the pool is skipped. Ids inside the pool must be
 *             distinct (repeated ids race; bros_check_slot_ids finds them).
 * Dense buffers k_out/v_out/k_in/v_in: [num_slots][num_kv_heads][head_dim] in
 * the pools' dtype, the layout of kv_write's new tokens. slot_ids: int32
 * [num_slots] device array. Bytes move unchanged (bit-exact).
 *
 * The dense buffers are device memory, or pinned host memory the device can
 * address (the kernel then runs at host-link speed and holds compute units
 * meanwhile). The intended use is a device staging buffer plus an
 * asynchronous copy on another stream: gather before the write that
 * overwrites the slots, then copy device-to-host while attention runs; copy
 * host-to-device ahead of time, then scatter before the attention that reads
 * the restored slots.
 *
 * Errors: BROS_E_NULL (a pointer NULL with num_slots > 0), BROS_E_SHAPE
 * (negative counts, num_blocks <= 0, num_kv_heads <= 0, misaligned tensors),
 * BROS_E_DTYPE, BROS_E_UNSUPPORTED (block_size != 16, head_dim != 128).
 * num_slots == 0 launches nothing.
 */
int bros_kv_gather(const void* k_pool, const void* v_pool, int32_t num_blocks,
                   const int32_t* slot_ids, int32_t num_slots,
                   void* k_out, void* v_out,
                   int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                   int32_t dtype, void* stream);
int bros_kv_scatter(const void* k_in, const void* v_in,
                    const int32_t* slot_ids, int32_t num_slots,
                    void* k_pool, void* v_pool, int32_t num_blocks,
                    int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                    int32_t dtype, void* stream);

/*
 * bros_copy_dma -- an asynchronous copy of `bytes` bytes on a copy (SDMA)
 * engine, ordered on `stream` like a kernel launched there.
 *
 * Defines: the host copies of Sec. 5.2's lazy checkpointing, carried on their
 * own streams (Sec. 6), so that they proceed beside kernels that occupy every
 * compute unit. The copy is handed to a copy engine through the ROCr runtime
 * that the HIP runtime has loaded, not to hipMemcpyAsync (whose engine choice
 * is the runtime's: the runtime bundled with PyTorch for ROCm 7.0 makes a copy
 * kernel of every such copy). The engine starts once the stream's earlier
 * work is done, and the stream's later work starts once the copy has landed:
 * two one-lane kernels on the stream release the engine and wait for it
 * through two HSA signals (the wait sleeps for the copy's shortest possible
 * duration and then polls every few microseconds); no host thread waits.
 * Host-to-device copies use one engine and device-to-host copies another, so
 * the two directions run at once (about 57 and 48 GB/s side by side on
 * MI355X, 56 GB/s alone).
 *
 * dst and src are device memory or pinned host memory (hipHostMalloc, or
 * torch's pin_memory), not both host; the ranges must not overlap; both stay
 * valid until the copy has ended on the stream. Copies on one engine run in
 * the order they were requested. Not for a stream under graph capture (the
 * engine copy would not be part of the graph). Returns BROS_OK, BROS_E_NULL
 * (a NULL pointer with bytes > 0), BROS_E_SHAPE (pageable host memory, or
 * both sides on the host), BROS_E_UNSUPPORTED (the stream is capturing) or
 * BROS_E_HIP (the runtime's entry points were not found, a call failed, or an
 * earlier copy's wait gave up after 10 s; if the stream could not take the
 * ordering kernels, the copy has been completed before the call returned).
 * Thread-safe.
 */
int bros_copy_dma(void* dst, const void* src, size_t bytes, void* stream);

/*
 * bros_check_slot_ids -- host-side check of a scatter's slot list: every id
 * inside [0, num_blocks * 16) appears once. slot_ids is a HOST pointer.
 * Returns BROS_OK or BROS_E_TABLE naming the first repeated id (BROS_E_NULL /
 * BROS_E_SHAPE for bad arguments).
 */
int bros_check_slot_ids(const int32_t* slot_ids, int32_t num_slots, int32_t num_blocks);

/*
 * bros_slot_ids -- slot ids of chosen (sequence, logical position) pairs.
 *
 * Defines: the slot mapping of Sec. 5.1 with the exclusive view of Sec. 5.2,
 * the one every kernel applies: position p of sequence s lives in block
 * block_tables[s][p / 16], slot p % 16 when its entry walks from the left
 * (+1) and 15 - p % 16 from the right (-1); the id is block * 16 + slot.
 * For i in [0, n): slot_ids[i] = id of (seqs[i], positions[i]). Directions
 * as in COMMON CONVENTIONS (dir per sequence, per table entry when
 * dir_per_entry is 1, or from cls when dir is NULL). All pointers are HOST
 * pointers; slot_ids is written by the caller-owned array of n entries.
 * Errors: BROS_E_NULL, BROS_E_SHAPE (bad counts), BROS_E_TABLE (a sequence
 * index outside [0, num_seqs), a position beyond the table, an entry outside
 * [0, num_blocks), a flag other than +1 / -1), naming the first bad pair.
 */
int bros_slot_ids(const int32_t* block_tables, int32_t max_blocks_per_seq, const int8_t* dir,
                  const uint8_t* cls, int32_t dir_per_entry, int32_t num_seqs, int32_t num_blocks,
                  const int32_t* seqs, const int32_t* positions, int32_t n, int32_t* slot_ids);

/*
 * bros_set_decode_kernel_events -- measurement hook for benchmarks.
 *
 * Not an operation of the paper: it lets a benchmark time the decode kernel
 * on its own, apart from the merge kernel that ends every bf16
 * bros_attn_decode call. With both events non-NULL (hipEvent_t handles, owned
 * by the caller, created with timing enabled), every following bf16
 * bros_attn_decode or bros_attn_decode_noalloc call records `before` on its
 * stream right before its decode kernel and `after` right after it, ahead of
 * the merge; hipEventElapsedTime(before, after) is then that kernel's
 * duration. NULL, NULL (the default) records nothing. The setting is
 * process-wide: set it from one thread, with no decode call in flight on
 * another. A failed record is reported by the decode call as BROS_E_HIP.
 * Returns BROS_OK, or BROS_E_NULL when exactly one event is NULL.
 */
int bros_set_decode_kernel_events(void* before, void* after);

/*
 * bros_stream_create_cu_share -- a stream whose kernels run on a fixed share
 * of the current device's compute units.
 *
 * Defines: the executor of Sec. 6 hands the prefill rows and the decode rows
 * of one batch to two different attention kernels. The first is bound by the
 * matrix cores and the second by HBM bandwidth; two such streams let them run
 * side by side on disjoint compute units (prefill on one share, decode on the
 * rest). bros_attn_decode sizes its grid by the compute units of the stream it
 * is given, so it fills a share exactly.
 *
 * The share is compute units [first_cu, first_cu + num_cus) in the order of a
 * HIP CU mask. On MI355X the runtime deals that order to the 8 dies in turn
 * and, within a die, to its 4 shader engines in turn, so a range whose start
 * and length are multiples of 32 holds the same number of compute units on
 * every die and engine. Other ranges are rejected (BROS_E_SHAPE): a grid
 * dispatched evenly over engines with unequal shares leaves work queued
 * behind the smaller ones. Also BROS_E_SHAPE: a range beyond the device's
 * compute units; BROS_E_NULL: stream is NULL; BROS_E_HIP: the runtime refused
 * the mask or applied a different one. On success *stream holds a new
 * hipStream_t at the default priority, owned by the caller, who releases it
 * with bros_stream_destroy; on failure *stream is NULL.
 */
int bros_stream_create_cu_share(int32_t first_cu, int32_t num_cus, void** stream);
/* Destroys a stream made by bros_stream_create_cu_share (after its work ends). */
int bros_stream_destroy(void* stream);

/*
 * bros_check_batch -- full host-side consistency check of a batch's metadata.
 *
 * Defines: the invariant behind Sec. 5.2 (two requests sharing a block never
 * own the same slot; a peer's token that would be overwritten is checkpointed
 * first, so a consistent batch maps distinct (sequence, position) pairs to
 * distinct (block, slot) pairs). All pointers are HOST pointers. Checks, in
 * order: counts and pointers, dir values in {+1, -1} (per sequence, or per
 * table entry below ceil(ctx / 16) when dir_per_entry is 1; cls in {RT, BE}
 * when dir is NULL), 0 <= ctx_lens[s] <= max_blocks_per_seq * 16, every referenced
 * table entry in [0, num_blocks), and -- when check_slot_disjointness != 0 --
 * that no (block, slot) is owned twice. Returns BROS_OK or BROS_E_TABLE (or
 * BROS_E_NULL / BROS_E_SHAPE / BROS_E_UNSUPPORTED) with a message naming the
 * first offending sequence and position.
 */
int bros_check_batch(const int32_t* block_tables, int32_t max_blocks_per_seq,
                     const int8_t* dir, const uint8_t* cls, int32_t dir_per_entry, const int32_t* ctx_lens,
                     int32_t num_seqs, int32_t num_blocks, int32_t block_size,
                     int32_t check_slot_disjointness);

/*
 * HOST BLOCK MANAGER AND SCHEDULER (host memory only; no GPU calls)
 *
 * Defines: Sec. 5.2 (Block Management): FindBlock places a request's KV in the
 * blocks with the most empty slots (a free block first); for RT requests
 * FindPreemptBlock takes BE blocks, again those with the most empty slots,
 * and writes from the opposite end; once a shared block's slots run out, only
 * the peer's tokens that a write would replace are saved first (lazy
 * checkpointing), the block enters the preemption table, and the tokens come
 * back when their request is scheduled again. Sec. 4.2: Alg. 1 (priority-
 * based packing) and adaptive batch sizing.
 *
 * Readings where the paper is silent: a request's entry e always holds its
 * positions [16 e, 16 e + 16) (the exclusive view); an RT token that meets a
 * BE token checkpoints it, while a BE token that meets an RT token moves the
 * BE entry to another block (BE never overwrites RT); a restored entry stays
 * in place when its missing slots are free, else it moves with its tokens.
 *
 * Ownership: a manager handle is created and destroyed by the caller; it is
 * not thread-safe. Plans name slots by id (block * 16 + slot).
 */
typedef struct bros_mgr_plan {
  int32_t* victims;      /* [victims_cap][4]: request, position, block, slot -- checkpoint BEFORE the write */
  int32_t victims_cap, num_victims;
  int32_t* move_src;     /* [moves_cap] slot ids: device moves (gather src -> scatter dst) BEFORE the write */
  int32_t* move_dst;
  int32_t moves_cap, num_moves;
  int32_t* restore_pos;  /* [restores_cap] positions of the request whose checkpointed rows come back */
  int32_t* restore_dst;  /* ... to these slot ids (after the moves) */
  int32_t restores_cap, num_restores;
  int32_t* written_pos;  /* [written_cap] position and slot id of every new token (grow only) */
  int32_t* written_slot;
  int32_t written_cap, num_written;
} bros_mgr_plan;

void* bros_mgr_create(int32_t num_blocks);                 /* NULL on error (bros_last_error) */
void bros_mgr_destroy(void* mgr);
int bros_mgr_add_request(void* mgr, int32_t req, int32_t cls);
int bros_mgr_release(void* mgr, int32_t req);             /* frees its slots; drops its checkpoints */
/* n_new more tokens for req (FindBlock / FindPreemptBlock, lazy checkpoints,
 * BE relocations). Fails with BROS_E_TABLE if req still has checkpointed
 * tokens (restore first) and BROS_E_NOMEM when blocks run out (tokens placed
 * before that stay placed and are reported in the plan). BROS_E_SHAPE if a
 * plan buffer is too small (the plan's counts give the sizes needed). */
int bros_mgr_grow(void* mgr, int32_t req, int32_t n_new, bros_mgr_plan* plan);
/* Brings req's checkpointed tokens back: moves and restore destinations. */
int bros_mgr_restore(void* mgr, int32_t req, bros_mgr_plan* plan);
/* One call for a whole iteration's block management: for i in [0, n), in
 * order, request reqs[i] is restored first when it has checkpointed tokens
 * (restore_first = 1; with 0 such a request fails with BROS_E_TABLE) and
 * then grown by n_new[i] tokens, as bros_mgr_restore and bros_mgr_grow do.
 * The plan holds every request's lists concatenated in request order; ends
 * (int32 [n][4], caller-owned) gives, after request i, the running counts of
 * victims, moves, restores and written tokens, so request i's entries of each
 * list are [ends[i-1][k], ends[i][k]). status[i] (int32 [n]) is BROS_OK or
 * that request's error (BROS_E_NOMEM, BROS_E_TABLE); a failing request keeps
 * what it placed before the failure and later requests still run. Returns
 * BROS_OK, the first request's error, BROS_E_SHAPE (an unknown request or a
 * negative count, checked before anything changes, or a plan buffer too
 * small) or BROS_E_NULL. Host memory only. */
int bros_mgr_grow_batch(void* mgr, const int32_t* reqs, const int32_t* n_new, int32_t n, int32_t restore_first,
                        bros_mgr_plan* plan, int32_t* ends, int32_t* status);
/* An entry count that every list of the plan of bros_mgr_grow_batch(reqs,
 * n_new, n) stays within (plan buffers of this many entries, victims 4 times
 * as many ints, never make it fail for want of room); -1 for bad arguments. */
int32_t bros_mgr_plan_bound(void* mgr, const int32_t* reqs, const int32_t* n_new, int32_t n);
int bros_mgr_query(void* mgr, int32_t req, int32_t* ctx, int32_t* num_entries, int32_t* checkpointed);
int bros_mgr_table(void* mgr, int32_t req, int32_t* out, int32_t cap);
int32_t bros_mgr_free_blocks(void* mgr);
/* Checks every internal invariant of the manager (owners and entries agree,
 * counts fit, block lists match block states); BROS_E_TABLE names the first
 * broken one. For tests and debugging; it walks every block. */
int bros_mgr_validate(void* mgr);
int32_t bros_mgr_available(void* mgr, int32_t cls);       /* blocks a new entry of class cls may take */
int32_t bros_mgr_entries_needed(void* mgr, int32_t req, int32_t n_new);
/* Preemption table: [n][3] (block, RT owner, BE owner) of blocks in preemption
 * status, up to cap rows; returns the total count. */
int32_t bros_mgr_preemption_table(void* mgr, int32_t* out, int32_t cap);

/* A queued request as Alg. 1 sees it. */
typedef struct bros_sched_req {
  int32_t id;
  int32_t prefill;       /* 1: prefill phase, 0: decode phase */
  int32_t n_new;         /* input tokens this iteration (Ln contribution) */
  int32_t ctx_after;     /* attended tokens after this iteration (La contribution) */
  double remaining_us;   /* RT: T_SLO - t_i - (k_i - 1) T_avg (sort key); BE: unused */
  int32_t m_cpu;         /* BE: checkpointed slots (sort key); RT: unused */
} bros_sched_req;

/* C(batch) of Sec. 4.1 per phase: coef[0] prefill, coef[1] decode, each
 * {a0, a1, b} in microseconds; per_request = 0 uses Ln * La, 1 uses the sum
 * of n_i * a_i as the interaction term. */
typedef struct bros_cost_model {
  double coef[2][3];
  int32_t per_request;
} bros_cost_model;

/* Alg. 1 for one iteration: RT requests by ascending remaining time while the
 * batch has room, blocks exist (FindPreemptBlock) and the estimated time stays
 * within the most urgent request's remaining time; then BE requests by
 * ascending m_cpu, packed while they fit, else replacing the least urgent
 * RT request. Writes the chosen ids (rt_ready / be_ready must hold n_rt /
 * n_be ids) and over_budget = 1 when the time budget stopped the RT loop. The
 * manager is only read. */
int bros_schedule(void* mgr, const bros_sched_req* rt, int32_t n_rt, const bros_sched_req* be, int32_t n_be,
                  int32_t batch_size, const bros_cost_model* cost, int32_t* rt_ready, int32_t* n_rt_ready,
                  int32_t* be_ready, int32_t* n_be_ready, int32_t* over_budget);
/* Alg. 1 with Sec. 4.2's request pulling: the RT queue comes as the pending
 * queue (any order) and the waiting queue, which the caller keeps in ascending
 * order of remaining time (the paper: the waiting queue is ordered by arrival,
 * so its head has waited longest). Only the pending queue is sorted, and only
 * its first batch_size requests (a partial sort); the RT order is then pulled
 * by polling the two queue heads and taking the more urgent one (pending
 * first on ties). The BE queue is partially sorted as far as the BE loop can
 * reach (2 batch_size + 1 requests). With a waiting queue in that order the
 * result equals bros_schedule over the pending and waiting requests together
 * (pending listed first). Same outputs and errors as bros_schedule. */
int bros_schedule_pulled(void* mgr, const bros_sched_req* pending, int32_t n_pending, const bros_sched_req* waiting,
                         int32_t n_waiting, const bros_sched_req* be, int32_t n_be, int32_t batch_size,
                         const bros_cost_model* cost, int32_t* rt_ready, int32_t* n_rt_ready, int32_t* be_ready,
                         int32_t* n_be_ready, int32_t* over_budget);
/* Adaptive batch sizing: back to `base` after an over-budget iteration, else
 * doubled (at most max_size). */
int32_t bros_next_batch_size(int32_t current, int32_t base, int32_t max_size, int32_t over_budget);

#ifdef __cplusplus
}
#endif

#endif /* BROS_ATTN_H */
