// bros_attn_prefill_chunk (bf16) launch on the matrix cores: the unit kernel
// and the merge of split units. The device code (and what it computes) is in
// prefill_device.h.
#include "prefill_device.h"

namespace bros {
namespace pf {

template <int G, bool kOff32>
__global__ __launch_bounds__(kThreads, 2) void prefill_mfma_kernel(PrefillArgs a) {
  BROS_PREFILL_UNIT_LDS
  prefill_unit<G, kOff32>(a, paired_id(a, blockIdx.x, gridDim.x), s_kring, s_vring, &s_first_bad, s_tbl, s_dir);
}

// Fold the pieces of split units: one workgroup per (split item, KV head),
// from the list the prefill grid's first workgroup wrote. Per row, with
// M = max_p m_p (log2 units): o = sum_p 2^(m_p - M) O_p / sum_p 2^(m_p - M) l_p.
// Rows of unsplit units were written by the prefill kernel itself.
template <int G>
__global__ __launch_bounds__(kThreads) void prefill_merge_kernel(PrefillArgs a) {
  constexpr int QT = kRows / G;
  __shared__ float s_m[kRows];
  __shared__ float s_inv[kRows];
  const int Hkv = a.num_kv_heads;
  const int j = blockIdx.x / Hkv, g = blockIdx.x % Hkv;
  if (j >= load_uniform(a.ws_list, 0)) return;
  const int item = load_uniform(a.ws_list, 1 + 3 * j);
  const int parts = load_uniform(a.ws_list, 2 + 3 * j);
  const int slot0 = load_uniform(a.ws_list, 3 + 3 * j);
  const int tps = a.tiles_per_seq;
  const int s = item / tps, t = item % tps;
  const int q_begin = load_uniform(a.cu_q, s);
  const int n = load_uniform(a.cu_q, s + 1) - q_begin;
  if (q_begin < 0 || n <= 0 || q_begin + n > a.num_q_tokens || t * QT >= n) return;   // (never split)
  const size_t row0 = ((size_t)slot0 * Hkv + g) * kRows;   // workspace row of part 0, unit row 0
  const size_t pstride = (size_t)Hkv * kRows;              // workspace rows from one part to the next
  const int tid = threadIdx.x;
  if (tid < kRows) {
    float m = -INFINITY;
    for (int p = 0; p < parts; ++p) m = fmaxf(m, a.ws_ml[2 * (row0 + p * pstride + tid)]);
    float l = 0.0f;
    for (int p = 0; p < parts; ++p) {
      const size_t row = row0 + p * pstride + tid;
      l = fmaf(a.ws_ml[2 * row + 1], fast_exp2(a.ws_ml[2 * row] - m), l);
    }
    s_m[tid] = m;
    s_inv[tid] = l > 0.0f ? 1.0f / l : 0.0f;
  }
  __syncthreads();
  const int c4 = tid & 31;   // dims 4 c4 .. 4 c4 + 3 of rows tid / 32 + 8 i
#pragma unroll 2
  for (int i = 0; i < kRows / 8; ++i) {
    const int r = 8 * i + (tid >> 5);
    const int qrow = t * QT + r % QT;
    if (qrow >= n) continue;
    const float m = s_m[r];
    float4 acc = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    for (int p = 0; p < parts; ++p) {
      const size_t row = row0 + p * pstride + r;
      const float w = fast_exp2(a.ws_ml[2 * row] - m);
      const float4 v = reinterpret_cast<const float4*>(a.ws_o + row * kHeadDim)[c4];
      acc.x = fmaf(v.x, w, acc.x);
      acc.y = fmaf(v.y, w, acc.y);
      acc.z = fmaf(v.z, w, acc.z);
      acc.w = fmaf(v.w, w, acc.w);
    }
    const float inv = s_inv[r];
    uint2 o2;
    o2.x = pack2_bf16(acc.x * inv, acc.y * inv);
    o2.y = pack2_bf16(acc.z * inv, acc.w * inv);
    const size_t orow = (size_t)(q_begin + qrow) * a.num_q_heads + g * G + r / QT;
    reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.out) + orow * kHeadDim)[c4] = o2;
  }
}

// Compute units a split plan spreads over, at most; the workspace holds
// 2 x this many (split piece, KV head) partials.
constexpr int kMaxPrefillCus = 512;

template <int G>
hipError_t launch_group(PrefillArgs a, int num_units, hipStream_t stream) {
  // Split only when the units leave compute units idle: with a unit or more
  // per compute unit, splitting measured no faster (its partials and merge
  // cost what the better balance saves).
  a.num_cus = 0;
  if (a.ws_o != nullptr && num_units / a.num_kv_heads <= kMaxRankItems) {
    int cus = stream_compute_units(stream);
    cus = cus < kMaxPrefillCus ? cus : kMaxPrefillCus;
    if (num_units < cus) a.num_cus = cus;
  }
  // Placement of the first round (two workgroups per compute unit): known
  // when the stream has the whole chip, so unsplit units are paired by work.
  a.xcd_cus = 0;
  if (a.num_cus == 0) {
    const int cus = stream_compute_units(stream);
    if (cus == stream_compute_units(nullptr) && cus % kXcds == 0) a.xcd_cus = cus / kXcds;
  }
  // ranks beyond the units: at most num_cus / Hkv more pieces than items
  const long long grid = (long long)num_units + a.num_cus;
  // (block, KV head) rows of 4 KiB: 32-bit offsets reach them all below 2^20 rows
  if ((int64_t)a.num_blocks * a.num_kv_heads <= (int64_t)1 << 20)
    hipLaunchKernelGGL((prefill_mfma_kernel<G, true>), dim3((unsigned)grid), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((prefill_mfma_kernel<G, false>), dim3((unsigned)grid), dim3(kThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.num_cus == 0) return e;
  // split items x Hkv <= num_cus
  hipLaunchKernelGGL(prefill_merge_kernel<G>, dim3((unsigned)a.num_cus), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace pf

using pf::kMaxPrefillCus;
using pf::kMaxRankItems;
using pf::kRows;
using pf::launch_group;

int prefill_positions_per_tile(int group) { return kRows / group; }

size_t prefill_workspace_bytes() {
  const size_t rows = 2 * (size_t)kMaxPrefillCus * kRows;   // (split piece, KV head) partials x rows
  const size_t bytes = rows * kHeadDim * sizeof(float) + rows * 2 * sizeof(float) + (1 + 3 * (size_t)kMaxRankItems) * sizeof(int32_t);
  return (bytes + 255) & ~(size_t)255;
}

void set_prefill_workspace(PrefillArgs& a, void* ws, size_t bytes) {
  a.num_cus = 0;
  a.ws_slots = 0;
  a.ws_o = nullptr;
  a.ws_ml = nullptr;
  a.ws_list = nullptr;
  if (ws == nullptr || bytes < prefill_workspace_bytes()) return;   // no splitting
  const size_t rows = 2 * (size_t)kMaxPrefillCus * kRows;
  a.ws_o = static_cast<float*>(ws);
  a.ws_ml = a.ws_o + rows * kHeadDim;
  a.ws_list = reinterpret_cast<int32_t*>(a.ws_ml + rows * 2);
  a.ws_slots = 2 * kMaxPrefillCus;
}

hipError_t launch_prefill_mfma(PrefillArgs a, int group, int num_tiles_total, hipStream_t stream) {
  if (num_tiles_total <= 0) return hipSuccess;
  switch (group) {
    case 1: return launch_group<1>(a, num_tiles_total, stream);
    case 2: return launch_group<2>(a, num_tiles_total, stream);
    case 4: return launch_group<4>(a, num_tiles_total, stream);
    case 8: return launch_group<8>(a, num_tiles_total, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace bros
