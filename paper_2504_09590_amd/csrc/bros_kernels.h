// Internal launch interface between the C ABI layer (api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace bros {

struct KvWriteArgs {
  const void* k_new;
  const void* v_new;
  void* k_pool;
  void* v_pool;
  const int32_t* block_tables;
  const int8_t* dir;
  const uint8_t* cls;
  const int32_t* pos0;
  const int32_t* cu_new;
  int32_t dir_per_entry;  // dir is [S][max_blocks_per_seq] (else [S])
  int32_t num_new_tokens;
  int32_t num_seqs;
  int32_t num_blocks;
  int32_t max_blocks_per_seq;
  int32_t num_kv_heads;
};

// Split-K decode over "query rows". In decode mode (cu_q == nullptr) row r is
// sequence r with context ctx_lens[r]. In row mode (cu_q != nullptr) row r is a
// prefill row of the sequence s with cu_q[s] <= r < cu_q[s+1] and sees the
// first ctx_lens[s] - (cu_q[s+1] - r) + 1 positions (causal, diagonal inclusive).
struct DecodeArgs {
  void* out;
  const void* q;
  const void* k_pool;
  const void* v_pool;
  const int32_t* block_tables;
  const int8_t* dir;
  const uint8_t* cls;
  const int32_t* ctx_lens;
  const int32_t* cu_q;
  int32_t dir_per_entry;  // dir is [S][max_blocks_per_seq] (else [S])
  // Partial results. fp32 split-K: [rows][Hq][n_split_max] slots. bf16 (one
  // worker per wave over an even share of the tiles): slot (row * Hkv + g +
  // worker) * G + head-in-group, for segments cut between workers.
  float* ws_acc;          // [slots][D] unnormalised partial outputs
  float* ws_ml;           // [slots][2] (running max in log2 units, sum)
  int32_t* ws_rows;       // bf16: first tile of each row, [rows + 1]
  int32_t* ws_cut;        // bf16: per worker, [2 w] the (row * Hkv + g) segment it starts and leaves cut, else -1;
                          // [2 w + 1] the worker holding that segment's last tile, or -1 if not computed
  int32_t* ws_wstart;     // bf16: [0] workers W, then [1 + w] first tile of worker w (w <= W)
  int32_t num_workers;    // bf16: waves of the grid (workers beyond the tile count idle)
  int32_t num_rows;
  int32_t num_seqs;
  int32_t num_blocks;
  int32_t max_blocks_per_seq;
  int32_t max_ctx;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t split_blocks;   // blocks per split, multiple of 4, <= 64
  int32_t n_split_max;
  float scale_log2;       // softmax scale * log2(e)
};

struct PrefillArgs {
  void* out;
  const void* q;
  const int32_t* cu_q;
  const void* k_pool;
  const void* v_pool;
  const int32_t* block_tables;
  const int8_t* dir;
  const uint8_t* cls;
  const int32_t* ctx_lens;
  int32_t dir_per_entry;  // dir is [S][max_blocks_per_seq] (else [S])
  int32_t num_q_tokens;
  int32_t num_seqs;
  int32_t num_blocks;
  int32_t max_blocks_per_seq;
  int32_t max_ctx;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t tiles_per_seq;  // ceil(max_q_len / positions per tile)
  float scale_log2;
  // Splitting long units into pieces over key ranges (none when num_cus is 0):
  // the compute units the work is spread over, the partials of split units,
  // [ws_slots][128 rows] x (ws_o: 128 dims, ws_ml: max and sum) in fp32, and
  // the list of split units that the merge walks (count, then (item, parts,
  // first slot) triples).
  int32_t num_cus;
  int32_t xcd_cus;        // compute units per XCD when the launch has the whole chip, else 0
  int32_t ws_slots;
  float* ws_o;
  float* ws_ml;
  int32_t* ws_list;
};

// Rows of a list of slots moved between the pool and a dense [n][Hkv][D]
// buffer (gather: pool -> dense, scatter: dense -> pool).
struct KvMoveArgs {
  void* k_pool;           // gather source / scatter destination (only read by the gather)
  void* v_pool;
  void* k_dense;          // gather destination / scatter source (only read by the scatter)
  void* v_dense;
  const int32_t* slot_ids;
  int32_t num_slots;
  int32_t num_blocks;
  int32_t num_kv_heads;
  int32_t row_bytes;      // head_dim * element bytes (a multiple of 16)
};

// Decode planning shared by the launcher and the workspace query.
struct DecodePlan {
  int32_t split_blocks;
  int32_t n_split_max;
};
DecodePlan plan_decode(int32_t num_rows, int32_t max_ctx);
size_t decode_workspace_bytes(int32_t num_rows, int32_t num_q_heads, int32_t max_ctx, bool bf16);
// Points the workspace fields of `a` (num_rows, num_q_heads, n_split_max set)
// into `ws`, laid out as decode_workspace_bytes sized it.
void set_decode_workspace(DecodeArgs& a, void* ws, bool bf16);

hipError_t launch_kv_write(const KvWriteArgs& a, bool bf16, hipStream_t stream);
hipError_t launch_kv_move(const KvMoveArgs& a, bool gather, hipStream_t stream);
hipError_t launch_decode(DecodeArgs a, int group, bool bf16, hipStream_t stream);
// Events the bf16 decode records around its decode kernel (both null: none).
void set_decode_kernel_events(hipEvent_t before, hipEvent_t after);
// Longest context the matrix-core prefill handles (its block table is staged
// whole in LDS); longer contexts take the vector path.
constexpr int32_t kPrefillMaxCtxMfma = 32768;
// Compute units enabled for `stream` (a stream made with
// hipExtStreamCreateWithCUMask runs on a subset of the device): the device's
// count is queried once per device, the stream's CU mask read on every call.
int stream_compute_units(hipStream_t stream);
// Workgroups of `kernel` (launched with `threads` threads) that the compute
// units enabled for `stream` hold at once; the per-CU occupancy is queried once
// per device and cache slot (0..7: bf16 decode 0..3, fp32 decode 4..7).
int resident_workgroups(const void* kernel, int threads, int slot, hipStream_t stream);

hipError_t launch_prefill_mfma(PrefillArgs a, int group, int num_tiles_total, hipStream_t stream);
// The merge of the bf16 decode's cut segments (after a decode or a fused launch).
hipError_t launch_decode_merge(const DecodeArgs& a, int group, hipStream_t stream);

// Expected times that place the decode work of a fused prefill|decode launch:
// a prefill unit costs unit_fixed_us + unit_tile_us per key tile on its
// workgroup, a decode tile decode_tile_us on one worker (wave). Every worker
// gets decode tiles in proportion to the time its workgroup has left after
// its prefill unit, so that all end together.
struct MixedModel {
  float unit_fixed_us;
  float unit_tile_us;
  float decode_tile_us;
};
// One launch over the concatenated batch (Sec. 6): workgroup b first runs
// prefill unit b of the matrix-core prefill (no splitting), then its waves
// take their share of the bf16 decode tiles; then the decode merge. pa is set
// up as for launch_prefill_mfma (its workspace fields unused), da as for
// launch_decode with its workspace. Returns hipErrorInvalidValue when the
// prefill units (num_units) exceed the grid or their items exceed what the
// planner ranks; the caller then runs the two calls in turn.
hipError_t launch_mixed(PrefillArgs pa, DecodeArgs da, MixedModel mm, int group, int num_units, hipStream_t stream);
int prefill_positions_per_tile(int group);
// Workspace of the matrix-core prefill (optional: without it no unit is split).
size_t prefill_workspace_bytes();
void set_prefill_workspace(PrefillArgs& a, void* ws, size_t bytes);

}  // namespace bros
