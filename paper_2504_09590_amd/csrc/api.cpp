// C ABI of the bidirectional paged-attention step: O(1) argument checks,
// launch planning, kernel launches, status strings. No per-call allocation,
// no synchronization, no state kept between calls.
#include "bros_attn.h"
#include "bros_error.h"
#include "bros_kernels.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <vector>

namespace {

using bros::fail;
using bros::ok;

bool aligned(const void* p, size_t n) { return (reinterpret_cast<uintptr_t>(p) % n) == 0; }

// Checks shared by the three entry points; sets *group on success.
int check_shapes(const char* fn, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                 int32_t block_size, int32_t dtype, int* group) {
  if (dtype != BROS_F32 && dtype != BROS_BF16) return fail(BROS_E_DTYPE, "%s: dtype %d is neither BROS_F32 nor BROS_BF16", fn, dtype);
  if (block_size != 16) return fail(BROS_E_UNSUPPORTED, "%s: block_size %d unsupported (16 only)", fn, block_size);
  if (head_dim != 128) return fail(BROS_E_UNSUPPORTED, "%s: head_dim %d unsupported (128 only)", fn, head_dim);
  if (num_kv_heads <= 0 || num_q_heads <= 0) return fail(BROS_E_SHAPE, "%s: head counts must be positive (Hq=%d Hkv=%d)", fn, num_q_heads, num_kv_heads);
  if (num_q_heads % num_kv_heads != 0) return fail(BROS_E_SHAPE, "%s: num_q_heads %d is not a multiple of num_kv_heads %d", fn, num_q_heads, num_kv_heads);
  const int g = num_q_heads / num_kv_heads;
  if (g != 1 && g != 2 && g != 4 && g != 8) return fail(BROS_E_UNSUPPORTED, "%s: group size %d unsupported (1, 2, 4 or 8)", fn, g);
  *group = g;
  return BROS_OK;
}

int check_meta(const char* fn, const void* block_tables, int32_t max_blocks_per_seq, const int8_t* dir,
               const uint8_t* cls, int32_t dir_per_entry, int32_t num_blocks) {
  if (block_tables == nullptr) return fail(BROS_E_NULL, "%s: block_tables is NULL", fn);
  if (dir == nullptr && cls == nullptr) return fail(BROS_E_NULL, "%s: dir and cls are both NULL", fn);
  if (dir_per_entry != 0 && dir_per_entry != 1) return fail(BROS_E_SHAPE, "%s: dir_per_entry %d is neither 0 nor 1", fn, dir_per_entry);
  if (dir_per_entry && dir == nullptr) return fail(BROS_E_NULL, "%s: dir_per_entry is set but dir is NULL", fn);
  if (max_blocks_per_seq <= 0) return fail(BROS_E_SHAPE, "%s: max_blocks_per_seq %d must be positive", fn, max_blocks_per_seq);
  if (num_blocks <= 0) return fail(BROS_E_SHAPE, "%s: num_blocks %d must be positive", fn, num_blocks);
  if (!aligned(block_tables, 4)) return fail(BROS_E_SHAPE, "%s: block_tables is not 4-byte aligned", fn);
  return BROS_OK;
}

// Compute units per step of a CU share: 8 dies x 4 shader engines.
constexpr int kCuShareGranule = 32;

int launch_status(const char* fn, hipError_t e) {
  if (e != hipSuccess) return fail(BROS_E_HIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
  return ok();
}

float resolve_scale(float scale, int head_dim) {
  const float s = scale > 0.0f ? scale : 1.0f / std::sqrt((float)head_dim);
  return s * 1.4426950408889634f;   // log2(e): the kernels use base-2 exponentials
}

}  // namespace

extern "C" {

int bros_kv_write(const void* k_new, const void* v_new, int32_t num_new_tokens,
                  void* k_pool, void* v_pool, int32_t num_blocks,
                  const int32_t* block_tables, int32_t max_blocks_per_seq,
                  const int8_t* dir, const uint8_t* cls, int32_t dir_per_entry,
                  const int32_t* pos0, const int32_t* cu_new,
                  int32_t num_seqs, int32_t num_kv_heads, int32_t head_dim,
                  int32_t block_size, int32_t dtype, void* stream) {
  const char* fn = "bros_kv_write";
  int group = 0;
  int st = check_shapes(fn, num_kv_heads, num_kv_heads, head_dim, block_size, dtype, &group);
  if (st) return st;
  if (num_new_tokens < 0 || num_seqs < 0) return fail(BROS_E_SHAPE, "%s: negative count (tokens=%d seqs=%d)", fn, num_new_tokens, num_seqs);
  // (a workgroup's chunk indices stay below 2^22, where the kernel's float quotient is exact)
  if (num_kv_heads > 16384) return fail(BROS_E_UNSUPPORTED, "%s: %d KV heads; at most 16384", fn, num_kv_heads);
  if (num_new_tokens == 0) return ok();
  if (num_seqs == 0) return fail(BROS_E_SHAPE, "%s: %d new tokens but no sequences", fn, num_new_tokens);
  if (!k_new || !v_new || !k_pool || !v_pool || !pos0 || !cu_new) return fail(BROS_E_NULL, "%s: a tensor or offset pointer is NULL", fn);
  st = check_meta(fn, block_tables, max_blocks_per_seq, dir, cls, dir_per_entry, num_blocks);
  if (st) return st;
  if (!aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(k_pool, 16) || !aligned(v_pool, 16))
    return fail(BROS_E_SHAPE, "%s: tensors must be 16-byte aligned", fn);
  bros::KvWriteArgs a{k_new, v_new, k_pool, v_pool, block_tables, dir, cls, pos0, cu_new, dir_per_entry,
                      num_new_tokens, num_seqs, num_blocks, max_blocks_per_seq, num_kv_heads};
  return launch_status(fn, bros::launch_kv_write(a, dtype == BROS_BF16, static_cast<hipStream_t>(stream)));
}

size_t bros_attn_workspace_size(int32_t kind, int32_t dtype, int32_t num_rows,
                                int32_t num_q_heads, int32_t head_dim, int32_t max_ctx) {
  if (num_rows <= 0 || num_q_heads <= 0 || head_dim != 128 || max_ctx < 0) return 0;
  if (dtype != BROS_F32 && dtype != BROS_BF16) return 0;
  const bool bf16 = dtype == BROS_BF16;
  if (kind == BROS_WS_DECODE) return bros::decode_workspace_bytes(num_rows, num_q_heads, max_ctx, bf16);
  if (kind == BROS_WS_PREFILL)
    return (bf16 && max_ctx <= bros::kPrefillMaxCtxMfma) ? bros::prefill_workspace_bytes()
                                                          : bros::decode_workspace_bytes(num_rows, num_q_heads, max_ctx, bf16);
  return 0;
}

int bros_attn_decode(void* out, const void* q,
                     const void* k_pool, const void* v_pool, int32_t num_blocks,
                     const int32_t* block_tables, int32_t max_blocks_per_seq,
                     const int8_t* dir, const uint8_t* cls, int32_t dir_per_entry, const int32_t* ctx_lens,
                     int32_t max_ctx, int32_t num_seqs, int32_t num_q_heads,
                     int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                     float scale, int32_t dtype, void* workspace, size_t workspace_bytes,
                     void* stream) {
  const char* fn = "bros_attn_decode";
  int group = 0;
  int st = check_shapes(fn, num_q_heads, num_kv_heads, head_dim, block_size, dtype, &group);
  if (st) return st;
  if (num_seqs < 0 || max_ctx < 0) return fail(BROS_E_SHAPE, "%s: negative count (seqs=%d max_ctx=%d)", fn, num_seqs, max_ctx);
  if (num_seqs == 0) return ok();
  if (!out || !q || !k_pool || !v_pool || !ctx_lens) return fail(BROS_E_NULL, "%s: a tensor or length pointer is NULL", fn);
  st = check_meta(fn, block_tables, max_blocks_per_seq, dir, cls, dir_per_entry, num_blocks);
  if (st) return st;
  if (!aligned(out, 16) || !aligned(q, 16) || !aligned(k_pool, 16) || !aligned(v_pool, 16))
    return fail(BROS_E_SHAPE, "%s: tensors must be 16-byte aligned", fn);
  const bool bf16 = dtype == BROS_BF16;
  if (bf16 && (long long)num_seqs * num_kv_heads * ((max_ctx + 15) / 16) > 0x7fffffffLL)
    return fail(BROS_E_SHAPE, "%s: more than 2^31 (row, KV head, block) tiles", fn);
  const size_t need = bros::decode_workspace_bytes(num_seqs, num_q_heads, max_ctx, bf16);
  if (need > 0 && (workspace == nullptr || workspace_bytes < need || !aligned(workspace, 16)))
    return fail(BROS_E_WORKSPACE, "%s: workspace of %zu bytes (16-byte aligned) required, got %zu at %p", fn, need, workspace_bytes, workspace);
  const bros::DecodePlan plan = bros::plan_decode(num_seqs, max_ctx);
  bros::DecodeArgs a{};
  a.out = out;
  a.q = q;
  a.k_pool = k_pool;
  a.v_pool = v_pool;
  a.block_tables = block_tables;
  a.dir = dir;
  a.cls = cls;
  a.dir_per_entry = dir_per_entry;
  a.ctx_lens = ctx_lens;
  a.cu_q = nullptr;
  a.num_rows = num_seqs;
  a.num_seqs = num_seqs;
  a.num_blocks = num_blocks;
  a.max_blocks_per_seq = max_blocks_per_seq;
  a.max_ctx = max_ctx;
  a.num_q_heads = num_q_heads;
  a.num_kv_heads = num_kv_heads;
  a.split_blocks = plan.split_blocks;
  a.n_split_max = plan.n_split_max;
  a.scale_log2 = resolve_scale(scale, head_dim);
  bros::set_decode_workspace(a, need > 0 ? workspace : nullptr, bf16);
  return launch_status(fn, bros::launch_decode(a, group, bf16, static_cast<hipStream_t>(stream)));
}

int bros_attn_prefill_chunk(void* out, const void* q, const int32_t* cu_q,
                            int32_t num_q_tokens, int32_t max_q_len,
                            const void* k_pool, const void* v_pool, int32_t num_blocks,
                            const int32_t* block_tables, int32_t max_blocks_per_seq,
                            const int8_t* dir, const uint8_t* cls, int32_t dir_per_entry, const int32_t* ctx_lens,
                            int32_t max_ctx, int32_t num_seqs, int32_t num_q_heads,
                            int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                            float scale, int32_t dtype, void* workspace, size_t workspace_bytes,
                            void* stream) {
  const char* fn = "bros_attn_prefill_chunk";
  int group = 0;
  int st = check_shapes(fn, num_q_heads, num_kv_heads, head_dim, block_size, dtype, &group);
  if (st) return st;
  if (num_seqs < 0 || num_q_tokens < 0 || max_q_len < 0 || max_ctx < 0)
    return fail(BROS_E_SHAPE, "%s: negative count (seqs=%d tokens=%d max_q_len=%d max_ctx=%d)", fn, num_seqs, num_q_tokens, max_q_len, max_ctx);
  if (num_seqs == 0 || num_q_tokens == 0) return ok();
  if (max_q_len == 0) return fail(BROS_E_SHAPE, "%s: max_q_len is 0 with %d query rows", fn, num_q_tokens);
  if (!out || !q || !cu_q || !k_pool || !v_pool || !ctx_lens) return fail(BROS_E_NULL, "%s: a tensor or length pointer is NULL", fn);
  st = check_meta(fn, block_tables, max_blocks_per_seq, dir, cls, dir_per_entry, num_blocks);
  if (st) return st;
  if (!aligned(out, 16) || !aligned(q, 16) || !aligned(k_pool, 16) || !aligned(v_pool, 16))
    return fail(BROS_E_SHAPE, "%s: tensors must be 16-byte aligned", fn);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const float scale_log2 = resolve_scale(scale, head_dim);

  if (dtype == BROS_BF16 && max_ctx <= bros::kPrefillMaxCtxMfma) {
    bros::PrefillArgs a{};
    a.out = out;
    a.q = q;
    a.cu_q = cu_q;
    a.k_pool = k_pool;
    a.v_pool = v_pool;
    a.block_tables = block_tables;
    a.dir = dir;
    a.cls = cls;
    a.dir_per_entry = dir_per_entry;
    a.ctx_lens = ctx_lens;
    a.num_q_tokens = num_q_tokens;
    a.num_seqs = num_seqs;
    a.num_blocks = num_blocks;
    a.max_blocks_per_seq = max_blocks_per_seq;
    a.max_ctx = max_ctx;
    a.num_q_heads = num_q_heads;
    a.num_kv_heads = num_kv_heads;
    const int qt = bros::prefill_positions_per_tile(group);
    a.tiles_per_seq = (max_q_len + qt - 1) / qt;
    a.scale_log2 = scale_log2;
    const long long total = (long long)num_seqs * num_kv_heads * a.tiles_per_seq;
    if (total > 0x7fffffffLL - 1024) return fail(BROS_E_SHAPE, "%s: grid of %lld workgroups too large", fn, total);
    // the workspace is optional here: with one of the queried size, long units are split
    if (aligned(workspace, 16)) bros::set_prefill_workspace(a, workspace, workspace_bytes);
    return launch_status(fn, bros::launch_prefill_mfma(a, group, (int)total, s));
  }

  // fp32 (and bf16 beyond the matrix-core path's context limit): every prefill
  // row is a decode row with its own causal context.
  const bool bf16 = dtype == BROS_BF16;
  if (bf16 && (long long)num_q_tokens * num_kv_heads * ((max_ctx + 15) / 16) > 0x7fffffffLL)
    return fail(BROS_E_SHAPE, "%s: more than 2^31 (row, KV head, block) tiles", fn);
  const size_t need = bros::decode_workspace_bytes(num_q_tokens, num_q_heads, max_ctx, bf16);
  if (need > 0 && (workspace == nullptr || workspace_bytes < need || !aligned(workspace, 16)))
    return fail(BROS_E_WORKSPACE, "%s: workspace of %zu bytes (16-byte aligned) required, got %zu at %p", fn, need, workspace_bytes, workspace);
  const bros::DecodePlan plan = bros::plan_decode(num_q_tokens, max_ctx);
  bros::DecodeArgs a{};
  a.out = out;
  a.q = q;
  a.k_pool = k_pool;
  a.v_pool = v_pool;
  a.block_tables = block_tables;
  a.dir = dir;
  a.cls = cls;
  a.dir_per_entry = dir_per_entry;
  a.ctx_lens = ctx_lens;
  a.cu_q = cu_q;
  a.num_rows = num_q_tokens;
  a.num_seqs = num_seqs;
  a.num_blocks = num_blocks;
  a.max_blocks_per_seq = max_blocks_per_seq;
  a.max_ctx = max_ctx;
  a.num_q_heads = num_q_heads;
  a.num_kv_heads = num_kv_heads;
  a.split_blocks = plan.split_blocks;
  a.n_split_max = plan.n_split_max;
  a.scale_log2 = scale_log2;
  bros::set_decode_workspace(a, need > 0 ? workspace : nullptr, bf16);
  return launch_status(fn, bros::launch_decode(a, group, bf16, s));
}

int bros_attn_mixed(void* out_prefill, const void* q_prefill, const int32_t* cu_q, int32_t num_q_tokens,
                    int32_t max_q_len, int32_t num_prefill_seqs, int32_t max_ctx_prefill,
                    void* out_decode, const void* q_decode, int32_t num_decode_seqs, int32_t max_ctx_decode,
                    const void* k_pool, const void* v_pool, int32_t num_blocks,
                    const int32_t* block_tables, int32_t max_blocks_per_seq,
                    const int8_t* dir, const uint8_t* cls, int32_t dir_per_entry, const int32_t* ctx_lens,
                    int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                    float scale, int32_t dtype, void* workspace, size_t workspace_bytes, void* stream) {
  const char* fn = "bros_attn_mixed";
  int group = 0;
  int st = check_shapes(fn, num_q_heads, num_kv_heads, head_dim, block_size, dtype, &group);
  if (st) return st;
  if (dtype != BROS_BF16) return fail(BROS_E_UNSUPPORTED, "%s: bf16 only (use the two calls for fp32)", fn);
  if (num_prefill_seqs < 0 || num_decode_seqs < 0 || num_q_tokens < 0 || max_q_len < 0 || max_ctx_prefill < 0 ||
      max_ctx_decode < 0)
    return fail(BROS_E_SHAPE, "%s: negative count", fn);
  if (max_ctx_prefill > bros::kPrefillMaxCtxMfma)
    return fail(BROS_E_UNSUPPORTED, "%s: prefill context %d beyond the matrix-core path's %d (use the two calls)", fn,
                max_ctx_prefill, bros::kPrefillMaxCtxMfma);
  if (!ctx_lens || !block_tables) return fail(BROS_E_NULL, "%s: ctx_lens or block_tables is NULL", fn);
  const int P = num_prefill_seqs, D = num_decode_seqs;
  const size_t tab_off = (size_t)P * max_blocks_per_seq;
  const int8_t* dir_d = dir ? dir + (dir_per_entry ? tab_off : (size_t)P) : nullptr;
  const uint8_t* cls_d = cls ? cls + P : nullptr;
  // one half only: its own call
  if (P == 0 || num_q_tokens == 0)
    return bros_attn_decode(out_decode, q_decode, k_pool, v_pool, num_blocks, block_tables + tab_off,
                            max_blocks_per_seq, dir_d, cls_d, dir_per_entry, ctx_lens + P, max_ctx_decode, D,
                            num_q_heads, num_kv_heads, head_dim, block_size, scale, dtype, workspace,
                            workspace_bytes, stream);
  if (D == 0)
    return bros_attn_prefill_chunk(out_prefill, q_prefill, cu_q, num_q_tokens, max_q_len, k_pool, v_pool, num_blocks,
                                   block_tables, max_blocks_per_seq, dir, cls, dir_per_entry, ctx_lens,
                                   max_ctx_prefill, P, num_q_heads, num_kv_heads, head_dim, block_size, scale, dtype,
                                   nullptr, 0, stream);
  // both halves: validate as the two calls do
  if (max_q_len == 0) return fail(BROS_E_SHAPE, "%s: max_q_len is 0 with %d query rows", fn, num_q_tokens);
  if (!out_prefill || !q_prefill || !cu_q || !out_decode || !q_decode || !k_pool || !v_pool)
    return fail(BROS_E_NULL, "%s: a tensor or offset pointer is NULL", fn);
  st = check_meta(fn, block_tables, max_blocks_per_seq, dir, cls, dir_per_entry, num_blocks);
  if (st) return st;
  if (!aligned(out_prefill, 16) || !aligned(q_prefill, 16) || !aligned(out_decode, 16) || !aligned(q_decode, 16) ||
      !aligned(k_pool, 16) || !aligned(v_pool, 16))
    return fail(BROS_E_SHAPE, "%s: tensors must be 16-byte aligned", fn);
  if ((long long)D * num_kv_heads * ((max_ctx_decode + 15) / 16) > 0x7fffffffLL)
    return fail(BROS_E_SHAPE, "%s: more than 2^31 decode (row, KV head, block) tiles", fn);
  const size_t need = bros::decode_workspace_bytes(D, num_q_heads, max_ctx_decode, true);
  if (workspace == nullptr || workspace_bytes < need || !aligned(workspace, 16))
    return fail(BROS_E_WORKSPACE, "%s: workspace of %zu bytes (16-byte aligned) required, got %zu at %p", fn, need,
                workspace_bytes, workspace);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const float scale_log2 = resolve_scale(scale, head_dim);

  bros::PrefillArgs pa{};
  pa.out = out_prefill;
  pa.q = q_prefill;
  pa.cu_q = cu_q;
  pa.k_pool = k_pool;
  pa.v_pool = v_pool;
  pa.block_tables = block_tables;
  pa.dir = dir;
  pa.cls = cls;
  pa.dir_per_entry = dir_per_entry;
  pa.ctx_lens = ctx_lens;
  pa.num_q_tokens = num_q_tokens;
  pa.num_seqs = P;
  pa.num_blocks = num_blocks;
  pa.max_blocks_per_seq = max_blocks_per_seq;
  pa.max_ctx = max_ctx_prefill;
  pa.num_q_heads = num_q_heads;
  pa.num_kv_heads = num_kv_heads;
  const int qt = bros::prefill_positions_per_tile(group);
  pa.tiles_per_seq = (max_q_len + qt - 1) / qt;
  pa.scale_log2 = scale_log2;
  const long long units = (long long)P * num_kv_heads * pa.tiles_per_seq;

  bros::DecodeArgs da{};
  da.out = out_decode;
  da.q = q_decode;
  da.k_pool = k_pool;
  da.v_pool = v_pool;
  da.block_tables = block_tables + tab_off;
  da.dir = dir_d;
  da.cls = cls_d;
  da.dir_per_entry = dir_per_entry;
  da.ctx_lens = ctx_lens + P;
  da.cu_q = nullptr;
  da.num_rows = D;
  da.num_seqs = D;
  da.num_blocks = num_blocks;
  da.max_blocks_per_seq = max_blocks_per_seq;
  da.max_ctx = max_ctx_decode;
  da.num_q_heads = num_q_heads;
  da.num_kv_heads = num_kv_heads;
  const bros::DecodePlan plan = bros::plan_decode(D, max_ctx_decode);
  da.split_blocks = plan.split_blocks;
  da.n_split_max = plan.n_split_max;
  da.scale_log2 = scale_log2;
  bros::set_decode_workspace(da, workspace, true);

  // Expected costs on MI355X, fitted to a per-workgroup timeline of this
  // launch on the mixed-step workload: a prefill unit ends at about 29 us +
  // 0.54 us per 32-key tile (its partner on the compute unit shares the
  // time), a decode tile takes 2.62 us on one wave. They only place work;
  // results do not depend on them.
  const bros::MixedModel mm{29.0f, 0.54f, 2.62f};
  const hipError_t e = units <= 0x7fffffffLL ? bros::launch_mixed(pa, da, mm, group, (int)units, s) : hipErrorInvalidValue;
  if (e != hipErrorInvalidValue) return launch_status(fn, e);
  // more prefill units than one grid holds: the two calls in turn
  st = bros_attn_prefill_chunk(out_prefill, q_prefill, cu_q, num_q_tokens, max_q_len, k_pool, v_pool, num_blocks,
                               block_tables, max_blocks_per_seq, dir, cls, dir_per_entry, ctx_lens, max_ctx_prefill, P,
                               num_q_heads, num_kv_heads, head_dim, block_size, scale, dtype, nullptr, 0, stream);
  if (st) return st;
  return bros_attn_decode(out_decode, q_decode, k_pool, v_pool, num_blocks, block_tables + tab_off,
                          max_blocks_per_seq, dir_d, cls_d, dir_per_entry, ctx_lens + P, max_ctx_decode, D,
                          num_q_heads, num_kv_heads, head_dim, block_size, scale, dtype, workspace, workspace_bytes,
                          stream);
}

static int kv_move(const char* fn, bool gather, void* k_pool, void* v_pool, int32_t num_blocks,
                   const int32_t* slot_ids, int32_t num_slots, void* k_dense, void* v_dense,
                   int32_t num_kv_heads, int32_t head_dim, int32_t block_size, int32_t dtype, void* stream) {
  int group = 0;
  int st = check_shapes(fn, num_kv_heads, num_kv_heads, head_dim, block_size, dtype, &group);
  if (st) return st;
  if (num_slots < 0) return fail(BROS_E_SHAPE, "%s: negative num_slots %d", fn, num_slots);
  if (num_slots == 0) return ok();
  if (num_blocks <= 0) return fail(BROS_E_SHAPE, "%s: num_blocks %d must be positive", fn, num_blocks);
  if (!k_pool || !v_pool || !k_dense || !v_dense || !slot_ids)
    return fail(BROS_E_NULL, "%s: a pool, dense buffer or slot_ids pointer is NULL", fn);
  if (!aligned(k_pool, 16) || !aligned(v_pool, 16) || !aligned(k_dense, 16) || !aligned(v_dense, 16) ||
      !aligned(slot_ids, 4))
    return fail(BROS_E_SHAPE, "%s: tensors must be 16-byte aligned", fn);
  bros::KvMoveArgs a{k_pool, v_pool, k_dense, v_dense, slot_ids, num_slots, num_blocks, num_kv_heads,
                     head_dim * (dtype == BROS_BF16 ? 2 : 4)};
  const hipError_t e = bros::launch_kv_move(a, gather, static_cast<hipStream_t>(stream));
  if (e == hipErrorInvalidValue) return fail(BROS_E_SHAPE, "%s: %d slots make a grid too large", fn, num_slots);
  return launch_status(fn, e);
}

int bros_kv_gather(const void* k_pool, const void* v_pool, int32_t num_blocks,
                   const int32_t* slot_ids, int32_t num_slots,
                   void* k_out, void* v_out,
                   int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                   int32_t dtype, void* stream) {
  return kv_move("bros_kv_gather", true, const_cast<void*>(k_pool), const_cast<void*>(v_pool), num_blocks,
                 slot_ids, num_slots, k_out, v_out, num_kv_heads, head_dim, block_size, dtype, stream);
}

int bros_kv_scatter(const void* k_in, const void* v_in,
                    const int32_t* slot_ids, int32_t num_slots,
                    void* k_pool, void* v_pool, int32_t num_blocks,
                    int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                    int32_t dtype, void* stream) {
  return kv_move("bros_kv_scatter", false, k_pool, v_pool, num_blocks, slot_ids, num_slots,
                 const_cast<void*>(k_in), const_cast<void*>(v_in), num_kv_heads, head_dim, block_size, dtype, stream);
}

int bros_set_decode_kernel_events(void* before, void* after) {
  if ((before == nullptr) != (after == nullptr))
    return fail(BROS_E_NULL, "bros_set_decode_kernel_events: give both events or neither");
  bros::set_decode_kernel_events(static_cast<hipEvent_t>(before), static_cast<hipEvent_t>(after));
  return ok();
}

int bros_stream_create_cu_share(int32_t first_cu, int32_t num_cus, void** stream) {
  const char* fn = "bros_stream_create_cu_share";
  if (stream == nullptr) return fail(BROS_E_NULL, "%s: stream is NULL", fn);
  *stream = nullptr;
  if (first_cu < 0 || num_cus <= 0 || first_cu % kCuShareGranule != 0 || num_cus % kCuShareGranule != 0)
    return fail(BROS_E_SHAPE, "%s: share [%d, %d + %d) must start and span multiples of %d compute units", fn,
                first_cu, first_cu, num_cus, kCuShareGranule);
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return fail(BROS_E_HIP, "%s: %s", fn, hipGetErrorString(e));
  if ((int64_t)first_cu + num_cus > cus)
    return fail(BROS_E_SHAPE, "%s: share [%d, %d) exceeds the device's %d compute units", fn, first_cu,
                first_cu + num_cus, cus);
  const size_t words = ((size_t)cus + 31) / 32;
  std::vector<uint32_t> want(words, 0u), got(words, 0u);
  for (int i = first_cu; i < first_cu + num_cus; ++i) want[i / 32] |= 1u << (i % 32);
  hipStream_t s = nullptr;
  e = hipExtStreamCreateWithCUMask(&s, (uint32_t)words, want.data());
  if (e != hipSuccess) return fail(BROS_E_HIP, "%s: hipExtStreamCreateWithCUMask: %s", fn, hipGetErrorString(e));
  e = hipExtStreamGetCUMask(s, (uint32_t)words, got.data());
  if (e != hipSuccess || got != want) {
    (void)hipStreamDestroy(s);
    return fail(BROS_E_HIP, "%s: the runtime applied a different CU mask (%s)", fn,
                e != hipSuccess ? hipGetErrorString(e) : "mask differs");
  }
  *stream = s;
  return ok();
}

int bros_stream_destroy(void* stream) {
  const char* fn = "bros_stream_destroy";
  if (stream == nullptr) return fail(BROS_E_NULL, "%s: stream is NULL", fn);
  const hipError_t e = hipStreamDestroy(static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(BROS_E_HIP, "%s: %s", fn, hipGetErrorString(e));
  return ok();
}

}  // extern "C"
