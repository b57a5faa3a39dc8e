// bros_attn_decode (bf16) launch: the decode kernel and the merge of cut
// segments. The device code (and what it computes) is in decode_device.h.
#include "decode_device.h"

#include <atomic>
#include <mutex>
#include <type_traits>

namespace bros {
namespace dm {

template <int G>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void decode_mfma_kernel(DecodeArgs a) {
  __shared__ int s_pre[kMaxRowsLds + 1];
  __shared__ int s_scan[kWaves];

  const int chunk = (a.num_rows + kMaxRowsLds - 1) / kMaxRowsLds;
  const int nch = (a.num_rows + chunk - 1) / chunk;
  const int total = build_tile_prefix(a, s_pre, s_scan, chunk, nch);

  // Each wave takes an equal share of the tiles; with fewer tiles than waves
  // the last waves idle, so every worker has at least one tile. Workgroup 0
  // records the partition for the merge.
  const int workers = min(a.num_workers, total);
  if (blockIdx.x == 0) {
    if (threadIdx.x == 0) a.ws_wstart[0] = workers;
    for (int w = threadIdx.x; w <= workers; w += kThreads)
      a.ws_wstart[1 + w] = (int)((int64_t)w * total / max(workers, 1));
  }
  const int wid = blockIdx.x * kWaves + wave_id_uniform();
  if (wid >= workers) {
    if (wid < a.num_workers && (threadIdx.x & (kWave - 1)) == 0) a.ws_cut[2 * wid] = -1;   // idle: nothing to merge
    return;
  }
  const int t0 = (int)((int64_t)wid * total / workers);
  const int t1 = (int)((int64_t)(wid + 1) * total / workers);
  decode_worker<G>(a, s_pre, chunk, nch, wid, t0, t1 - t0, total, workers);
}

// Segments cut between workers: o = sum_w 2^(m_w - M) acc_w / sum_w 2^(m_w -
// M) l_w over the partials of workers w0 .. w1. The decode kernel's worker
// w0 (the one that started the segment and left it unfinished) named the
// segment in its entry of the cut list, with w1 when its shares are the even
// split (then every worker has tiles and the merge reads nothing else before
// the partials); every other entry is -1, so the merge grid has one wave per
// worker and most waves return after one load. Segments
// a single worker covered were written directly, and rows without context
// were written as zeros by that worker (a worker that sees no tile of a row
// never runs for it: rows without context have no tiles, so they are written
// here). The G heads of the segment share the wave: 64 / G lanes per head,
// each folding 2 G of its head's dims, eight partials in flight. (Merging
// inside the decode kernel instead would need device-scope release/acquire
// between workgroups, which on this chip writes back and invalidates a whole
// L2 per segment; the kernel boundary is far cheaper.)
constexpr int kMergeWaves = 4;

template <int G>
__global__ __launch_bounds__(kMergeWaves * kWave) void decode_mfma_merge_kernel(DecodeArgs a) {
  constexpr int L = kWave / G;          // lanes per head
  constexpr int DPL = kHeadDim / L;     // dims per lane (2 G)
  const int lane = threadIdx.x & (kWave - 1);
  const int item = blockIdx.x * kMergeWaves + wave_id_uniform();
  // Rows without context have no tiles, so no worker saw them: zeros.
  if (item < a.num_rows) {
    int s0, ctx0;
    resolve_row(a, item, s0, ctx0);
    if (ctx0 <= 0) {
      uint32_t* z = reinterpret_cast<uint32_t*>(static_cast<uint16_t*>(a.out) + (size_t)item * a.num_q_heads * kHeadDim);
      for (int i = lane; i < a.num_q_heads * kHeadDim / 2; i += kWave) z[i] = 0u;
    }
  }
  // every worker of the grid wrote its cut-list entry (idle ones -1)
  if (item >= a.num_workers) return;
  const int code = a.ws_cut[2 * item];
  if (code < 0) return;
  const int nkv = a.num_kv_heads;
  const int row = __builtin_amdgcn_readfirstlane(code / nkv);
  const int g = __builtin_amdgcn_readfirstlane(code - (code / nkv) * nkv);
  const int w0 = item;
  int w1 = __builtin_amdgcn_readfirstlane(a.ws_cut[2 * item + 1]);
  // the decode grid's partition of the tiles: workers W, worker w's tiles
  // start at starts[w] (starts[W] = all tiles); a worker may have none, but
  // not under the even split (w1 given)
  const int32_t* starts = a.ws_wstart + 1;
  const bool even = w1 >= 0;
  if (!even) {
    // w1: the worker holding the segment's last tile (the last worker whose
    // share starts at or before it), found 64 workers per step
    const int workers = a.ws_wstart[0];
    int s, ctx;
    resolve_row(a, row, s, ctx);
    const int nblk = (ctx + kBlockSize - 1) / kBlockSize;
    const int64_t last_tile = (int64_t)a.ws_rows[row] + (int64_t)g * nblk + nblk - 1;
    w1 = w0;
    for (int base = w0 + 1; base < workers; base += kWave) {
      const int w = base + lane;
      const bool before = w < workers && starts[w] <= last_tile;
      const uint64_t m = __builtin_amdgcn_ballot_w64(before);
      w1 = base + __builtin_popcountll(m) - 1;
      if (m != ~0ull) break;
    }
    w1 = __builtin_amdgcn_readfirstlane(max(w1, w0));
  }
  // a worker with no tiles wrote no partial
  auto has_tiles = [&](int w) -> bool { return even || starts[w + 1] > starts[w]; };
  const int hl = lane / L, sub = lane % L;
  const size_t seg = (size_t)row * nkv + g;
  float Lsum = 0.0f, M = kNoMax;
  float acc[DPL];
#pragma unroll
  for (int d = 0; d < DPL; ++d) acc[d] = 0.0f;
  // Fold partials c + u, u < cnt <= 8, of the head: lane j0 + u of the head's
  // lanes holds partial c + u's weight in wt and whether its worker had tiles
  // (and so wrote it) in ok; v[u] holds partial c + u's dims of this lane.
  // Padding and partials of workers without tiles add zero: their slots may
  // hold anything.
  auto fold8 = [&](int cnt, int j0, const float2 (&v)[8][DPL / 2], float wt, int ok) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = j0 + min(u, cnt - 1);
      const float w = __shfl(wt, hl * L + j);
      const bool use = u < cnt && __shfl(ok, hl * L + j) != 0;
      const float wu = use ? w : 0.0f;
#pragma unroll
      for (int q = 0; q < DPL / 2; ++q) {
        const float2 x = use ? v[u][q] : make_float2(0.0f, 0.0f);
        acc[2 * q] = fmaf(x.x, wu, acc[2 * q]);
        acc[2 * q + 1] = fmaf(x.y, wu, acc[2 * q + 1]);
      }
    }
  };
  auto load8 = [&](int c, int cnt, float2 (&v)[8][DPL / 2]) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {   // indices clamped in range
      const int j = min(u, cnt - 1);
      const float2* src = reinterpret_cast<const float2*>(a.ws_acc + ((seg + c + j) * G + hl) * kHeadDim + sub * DPL);
#pragma unroll
      for (int q = 0; q < DPL / 2; ++q) v[u][q] = src[q];
    }
  };
  if (w1 - w0 < 8) {
    // Up to eight partials (the common case): their sums are requested
    // together with their maxima, in one round of loads.
    const int cnt = w1 - w0 + 1;
    float2 v[8][DPL / 2];
    load8(w0, cnt, v);
    const int ok = sub < cnt && has_tiles(w0 + sub);
    float m_l = kNoMax, l_l = 0.0f;
    if (ok) {
      const size_t slot = (seg + w0 + sub) * G + hl;
      m_l = a.ws_ml[2 * slot];
      l_l = a.ws_ml[2 * slot + 1];
    }
    M = fmaxf(M, m_l);
#pragma unroll
    for (int o = L / 2; o >= 1; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
    float wt = 0.0f;
    if (ok) {
      wt = fast_exp2(m_l - M);
      Lsum = fmaf(l_l, wt, Lsum);
    }
    fold8(cnt, 0, v, wt, ok);
  } else {
    // the head's max over the partials (lanes of the head take every L-th one)
    for (int w = w0 + sub; w <= w1; w += L)
      if (has_tiles(w)) M = fmaxf(M, a.ws_ml[2 * ((seg + w) * G + hl)]);
#pragma unroll
    for (int o = L / 2; o >= 1; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
    for (int c = w0; c <= w1; c += L) {
      // lane sub holds the weight of partial c + sub of its head
      float wt = 0.0f;
      const int ok = c + sub <= w1 && has_tiles(c + sub);
      if (ok) {
        const size_t slot = (seg + c + sub) * G + hl;
        wt = fast_exp2(a.ws_ml[2 * slot] - M);
        Lsum = fmaf(a.ws_ml[2 * slot + 1], wt, Lsum);
      }
      const int cnt = min(L, w1 - c + 1);
      for (int j0 = 0; j0 < cnt; j0 += 8) {
        float2 v[8][DPL / 2];
        load8(c + j0, min(8, cnt - j0), v);
        fold8(min(8, cnt - j0), j0, v, wt, ok);
      }
    }
  }
#pragma unroll
  for (int o = L / 2; o >= 1; o >>= 1) Lsum += __shfl_xor(Lsum, o);
  const float inv = Lsum > 0.0f ? 1.0f / Lsum : 0.0f;
  uint32_t* out = reinterpret_cast<uint32_t*>(static_cast<uint16_t*>(a.out) +
                                              ((size_t)row * a.num_q_heads + g * G + hl) * kHeadDim + sub * DPL);
#pragma unroll
  for (int d = 0; d < DPL; d += 2) out[d / 2] = pack2_bf16(acc[d] * inv, acc[d + 1] * inv);
}

}  // namespace dm

namespace {

// Compute units enabled for `stream`: the population count of its CU mask, or
// `fallback` when the mask cannot be read.
int stream_cus(hipStream_t stream, int fallback) {
  constexpr int kMaskWords = 32;   // up to 1024 CUs
  uint32_t mask[kMaskWords] = {};
  if (hipExtStreamGetCUMask(stream, kMaskWords, mask) != hipSuccess) {
    (void)hipGetLastError();
    return fallback;
  }
  int n = 0;
  for (int i = 0; i < kMaskWords; ++i) n += __builtin_popcount(mask[i]);
  return (n > 0 && n < fallback) ? n : fallback;
}

}  // namespace

int stream_compute_units(hipStream_t stream) {
  constexpr int kMaxDevices = 64;
  static int cus_cache[kMaxDevices];
  static std::mutex mu;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
  int cus = 0;
  {
    std::lock_guard<std::mutex> lock(mu);
    if (cus_cache[dev] == 0) {
      int n = 0;
      if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
      cus_cache[dev] = n;
    }
    cus = cus_cache[dev];
  }
  return stream_cus(stream, cus);
}

int resident_workgroups(const void* kernel, int threads, int slot, hipStream_t stream) {
  constexpr int kMaxDevices = 64;
  constexpr int kSlots = 8;
  static int per_cu_cache[kMaxDevices][kSlots];
  static std::mutex mu;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 1024;
  int per_cu = 0;
  {
    std::lock_guard<std::mutex> lock(mu);
    if (per_cu_cache[dev][slot] == 0) {
      int n = 0;
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, threads, 0) != hipSuccess || n <= 0) n = 4;
      per_cu_cache[dev][slot] = n;
    }
    per_cu = per_cu_cache[dev][slot];
  }
  return per_cu * stream_compute_units(stream);
}

namespace {

// Workgroups of the bf16 decode grid at most (four workers each): what 256
// compute units hold at four waves per SIMD (the kernel runs two). The
// workspace is sized for it.
constexpr int kMaxDecodeGrid = 1024;

// Events recorded around the decode kernel of every bf16 call (a
// benchmark's hook; both null when unused).
std::atomic<hipEvent_t> g_kernel_ev_before{nullptr}, g_kernel_ev_after{nullptr};

template <int G>
hipError_t launch_group(DecodeArgs a, hipStream_t stream, int slot) {
  int grid = resident_workgroups(reinterpret_cast<const void*>(&dm::decode_mfma_kernel<G>), kThreads, slot, stream);
  grid = grid < kMaxDecodeGrid ? grid : kMaxDecodeGrid;
  a.num_workers = grid * kWaves;
  const hipEvent_t before = g_kernel_ev_before.load(), after = g_kernel_ev_after.load();
  hipError_t e = hipSuccess;
  if (before != nullptr && (e = hipEventRecord(before, stream)) != hipSuccess) return e;
  hipLaunchKernelGGL((dm::decode_mfma_kernel<G>), dim3(grid), dim3(kThreads), 0, stream, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (after != nullptr && (e = hipEventRecord(after, stream)) != hipSuccess) return e;
  return launch_decode_merge(a, G, stream);
}

}  // namespace

hipError_t launch_decode_merge(const DecodeArgs& a, int group, hipStream_t stream) {
  // one wave per worker (its cut-list entry) and per row (rows without context)
  const long long items = a.num_workers > a.num_rows ? a.num_workers : a.num_rows;
  const dim3 grid((unsigned)((items + dm::kMergeWaves - 1) / dm::kMergeWaves)), block(dm::kMergeWaves * kWave);
  switch (group) {
    case 1: hipLaunchKernelGGL(dm::decode_mfma_merge_kernel<1>, grid, block, 0, stream, a); break;
    case 2: hipLaunchKernelGGL(dm::decode_mfma_merge_kernel<2>, grid, block, 0, stream, a); break;
    case 4: hipLaunchKernelGGL(dm::decode_mfma_merge_kernel<4>, grid, block, 0, stream, a); break;
    case 8: hipLaunchKernelGGL(dm::decode_mfma_merge_kernel<8>, grid, block, 0, stream, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

DecodePlan plan_decode(int32_t num_rows, int32_t max_ctx) {
  DecodePlan p;
  const int64_t maxblk = max_ctx > 0 ? ((int64_t)max_ctx + kBlockSize - 1) / kBlockSize : 1;
  int sb = dm::kMaxSplitBlocks;   // 1024 tokens per split by default
  while (sb > 4 && (int64_t)num_rows * ((maxblk + sb - 1) / sb) < 512) sb >>= 1;
  p.split_blocks = sb;
  p.n_split_max = (int32_t)((maxblk + sb - 1) / sb);
  return p;
}

static size_t round_up_256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t decode_workspace_bytes(int32_t num_rows, int32_t num_q_heads, int32_t max_ctx, bool bf16) {
  if (bf16) {
    const int gmax = num_q_heads < 8 ? num_q_heads : 8;
    const size_t slots = (size_t)num_rows * num_q_heads + (size_t)kWaves * kMaxDecodeGrid * gmax;
    return round_up_256(((size_t)num_rows + 1) * sizeof(int32_t)) + round_up_256(slots * kHeadDim * sizeof(float)) +
           round_up_256(slots * 2 * sizeof(float)) + round_up_256((size_t)2 * kWaves * kMaxDecodeGrid * sizeof(int32_t)) +
           round_up_256(((size_t)kWaves * kMaxDecodeGrid + 2) * sizeof(int32_t));
  }
  const DecodePlan p = plan_decode(num_rows, max_ctx);
  if (p.n_split_max <= 1) return 0;
  const size_t slots = (size_t)num_rows * num_q_heads * p.n_split_max;
  return slots * kHeadDim * sizeof(float) + slots * 2 * sizeof(float);
}

void set_decode_workspace(DecodeArgs& a, void* ws, bool bf16) {
  char* base = static_cast<char*>(ws);
  if (bf16) {
    const int gmax = a.num_q_heads < 8 ? a.num_q_heads : 8;
    const size_t slots = (size_t)a.num_rows * a.num_q_heads + (size_t)kWaves * kMaxDecodeGrid * gmax;
    a.ws_rows = reinterpret_cast<int32_t*>(base);
    a.ws_acc = reinterpret_cast<float*>(base + round_up_256(((size_t)a.num_rows + 1) * sizeof(int32_t)));
    a.ws_ml = reinterpret_cast<float*>(reinterpret_cast<char*>(a.ws_acc) + round_up_256(slots * kHeadDim * sizeof(float)));
    a.ws_cut = reinterpret_cast<int32_t*>(reinterpret_cast<char*>(a.ws_ml) + round_up_256(slots * 2 * sizeof(float)));
    a.ws_wstart = reinterpret_cast<int32_t*>(reinterpret_cast<char*>(a.ws_cut) +
                                             round_up_256((size_t)2 * kWaves * kMaxDecodeGrid * sizeof(int32_t)));
    return;
  }
  a.ws_rows = nullptr;
  a.ws_cut = nullptr;
  a.ws_wstart = nullptr;
  a.ws_acc = reinterpret_cast<float*>(base);
  a.ws_ml = base ? a.ws_acc + (size_t)a.num_rows * a.num_q_heads * a.n_split_max * kHeadDim : nullptr;
}

void set_decode_kernel_events(hipEvent_t before, hipEvent_t after) {
  g_kernel_ev_before.store(before);
  g_kernel_ev_after.store(after);
}

hipError_t launch_decode(DecodeArgs a, int group, bool bf16, hipStream_t stream) {
  if (!bf16) return launch_decode_f32(a, group, stream);
  switch (group) {
    case 1: return launch_group<1>(a, stream, 0);
    case 2: return launch_group<2>(a, stream, 1);
    case 4: return launch_group<4>(a, stream, 2);
    case 8: return launch_group<8>(a, stream, 3);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace bros
