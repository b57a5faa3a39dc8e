// One launch over a mixed batch: the prefill chunks and the decode rows of the
// concatenated batch of Sec. 6 (prefill requests along the token axis with a
// length table, decode requests after them) in a single grid.
//
// The two halves cannot share a compute unit at the same time here: at two
// waves per SIMD the decode fills 2 x 181 of a SIMD's 512 registers and a
// prefill wave needs 210, and the decode loses a third of its rate with one
// wave per SIMD (measured), so a third, smaller prefill wave per SIMD is the
// only way to co-reside and the decode cannot afford it. What one launch
// does gain is the prefill's tail: its units differ in length, so compute
// units finish their prefill at different times (38-54 us on the mixed
// step). Here every workgroup (two per compute unit, four waves) first runs
// one prefill unit, exactly as the prefill kernel does, and then its waves
// take decode tiles; each worker's share is sized by the time its workgroup
// has left after its unit, so that workgroups with short units take more
// decode work and all end together. The prefill's kernel boundary goes too.
//
// Placement of the decode work: workgroup b expects its unit to take
// e_b = unit_fixed_us + unit_tile_us * L_b (0 without a unit), and a worker
// decode_tile_us per decode tile. With W workers and T decode tiles, all end
// at E = (decode_tile_us * T + sum_w e_w) / W when worker w takes
// (E - e_w) / decode_tile_us tiles (workers with e_w > E take none, and E is
// taken again over the others). Every workgroup computes the same partition
// from the same lengths in the same order; contiguous ranges in (row, KV
// head, block) order as in the decode kernel, so the partial slots and the
// merge are the decode's. The times are estimates: they only move work
// between workers, never change a result.
#include "decode_device.h"
#include "prefill_device.h"

namespace bros {
namespace {

constexpr int kThreadsMixed = 256;   // four waves, as both halves use
constexpr int kWavesMixed = kThreadsMixed / kWave;
static_assert(kThreadsMixed == pf::kThreads && kThreadsMixed == kThreads, "one workgroup shape for both halves");
// decode tile prefix in the K ring's LDS: (rows + 1) + one scan slot per thread
static_assert((kMaxRowsLds + 1 + kThreadsMixed) * sizeof(int) <= pf::kSlots * pf::kTileBytes, "prefix fits the ring");

template <int G, bool kOff32>
__global__ __launch_bounds__(kThreadsMixed, 2) void mixed_kernel(PrefillArgs pa, DecodeArgs da, MixedModel mm) {
  BROS_PREFILL_UNIT_LDS
  const int tid = threadIdx.x;
  const int grid = gridDim.x;
  constexpr int QT = pf::kRows / G;

  // ---- 1. this workgroup's prefill unit (none past the last rank)
  pf::prefill_unit<G, kOff32>(pa, pf::paired_id(pa, blockIdx.x, grid), s_kring, s_vring, &s_first_bad, s_tbl, s_dir);
  __syncthreads();   // the rings are free again

  // ---- 2. the decode's tile prefix over rows, in the K ring
  int* s_pre = reinterpret_cast<int*>(s_kring);
  int* s_scan = s_pre + kMaxRowsLds + 1;
  const int chunk = (da.num_rows + kMaxRowsLds - 1) / kMaxRowsLds;
  const int nch = (da.num_rows + chunk - 1) / chunk;
  const int total = dm::build_tile_prefix(da, s_pre, s_scan, chunk, nch);

  // ---- 3. every workgroup's expected prefill time: unit lengths ranked
  // longest first, as the units were handed out (V ring as scratch)
  int* s_sorted = reinterpret_cast<int*>(s_vring);                 // [kMaxRankItems] length of rank r
  float* s_cap = reinterpret_cast<float*>(s_sorted + pf::kMaxRankItems);   // [grid] decode tiles per worker
  double* s_red = reinterpret_cast<double*>(s_cap + 1024);              // [kWavesMixed] reduction slots
  const int tps = pa.tiles_per_seq;
  const int n_items = pa.num_seqs * tps;   // <= kMaxRankItems (checked by the launch)
  const int Hkv = pa.num_kv_heads;
  if (tid < n_items) {
    const int L = pf::unit_tiles(pa, tid / tps, tid % tps, QT);
    s_cap[tid] = (float)L;   // (borrowed for the lengths)
  }
  __syncthreads();
  if (tid < n_items) {
    const float mine = s_cap[tid];
    int r = 0;
    for (int j = 0; j < n_items; ++j) {
      const float lj = s_cap[j];
      r += (lj > mine) | ((lj == mine) & (j < tid));
    }
    s_sorted[r] = (int)mine;
  }
  __syncthreads();
  // e_b of workgroups tid and tid + 256, ... ; sums in a fixed order
  auto expected = [&](int b) -> float {
    const int rank = pf::paired_id(pa, b, grid) / Hkv;
    const int L = rank < n_items ? s_sorted[rank] : 0;
    return L > 0 ? mm.unit_fixed_us + mm.unit_tile_us * (float)L : 0.0f;
  };
  auto block_sum = [&](double v) -> double {   // the same order on every workgroup
#pragma unroll
    for (int o = kWave / 2; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    __syncthreads();
    if ((tid & (kWave - 1)) == 0) s_red[tid / kWave] = v;
    __syncthreads();
    double t = 0.0;
    for (int i = 0; i < kWavesMixed; ++i) t += s_red[i];
    return t;
  };
  const double rho = mm.decode_tile_us;
  // E over the workgroups whose unit ends before it (two passes)
  double E = 0.0;
  {
    double se = 0.0;
    for (int b = tid; b < grid; b += kThreadsMixed) se += expected(b);
    const double sum_e = block_sum(se);
    E = (rho * total + kWavesMixed * sum_e) / ((double)kWavesMixed * grid);
    double se2 = 0.0, cnt = 0.0;
    for (int b = tid; b < grid; b += kThreadsMixed) {
      const double e = expected(b);
      if (e <= E) {
        se2 += e;
        cnt += 1.0;
      }
    }
    const double sum_e2 = block_sum(se2), n2 = block_sum(cnt);
    if (n2 > 0.0) E = (rho * total + kWavesMixed * sum_e2) / (kWavesMixed * n2);
  }
  for (int b = tid; b < grid; b += kThreadsMixed) s_cap[b] = (float)fmax(0.0, (E - expected(b)) / rho);
  __syncthreads();
  // Whole tiles per workgroup, summing to the total exactly: each gets the
  // floor of its share, and the first (total - sum of floors) one more. Then
  // an exact integer prefix; integers keep every range consistent between
  // the workers and the table the merge reads.
  int* s_q = reinterpret_cast<int*>(s_red + kWavesMixed);   // [grid] tiles of workgroup b
  int* s_off = s_q + 1024;                                  // [grid + 1] first tile of workgroup b
  double cs = 0.0;
  for (int b = tid; b < grid; b += kThreadsMixed) cs += s_cap[b];
  const double cap_total = block_sum(cs);
  double qs = 0.0;
  for (int b = tid; b < grid; b += kThreadsMixed) {
    // (equal shares if no workgroup had time left, which the choice of E rules out)
    const double share = cap_total > 0.0 ? s_cap[b] / cap_total : 1.0 / grid;
    const int q = (int)fmin((double)total, floor((double)total * share));
    s_q[b] = q;
    qs += q;
  }
  const int rem = total - (int)block_sum(qs);   // 0 <= rem < grid (each floor loses less than one)
  for (int b = tid; b < grid; b += kThreadsMixed) s_q[b] += b < rem ? 1 : 0;
  __syncthreads();
  if (tid < kWave) {   // one wave: exclusive prefix over the workgroups, 64 at a time
    int carry = 0;
    for (int base = 0; base < grid; base += kWave) {
      const int b = base + tid;
      const int v = b < grid ? s_q[b] : 0;
      int inc = v;
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        const int u = __shfl_up(inc, o);
        if (tid >= o) inc += u;
      }
      if (b < grid) s_off[b] = carry + inc - v;
      carry += __shfl(inc, kWave - 1);
    }
    if (tid == 0) s_off[grid] = carry;
  }
  __syncthreads();
  const int W = grid * kWavesMixed;
  // first tile of worker k of workgroup b: the workgroup's tiles split evenly
  auto first_tile = [&](int b, int k) -> int { return s_off[b] + (int)((int64_t)s_q[b] * k / kWavesMixed); };
  if (blockIdx.x == 0) {
    // the partition for the merge: worker count, then every worker's first tile
    if (tid == 0) da.ws_wstart[0] = W;
    for (int w = tid; w <= W; w += kThreadsMixed)
      da.ws_wstart[1 + w] = w == W ? s_off[grid] : first_tile(w / kWavesMixed, w % kWavesMixed);
  }

  // ---- 4. this wave's decode tiles
  const int wave = wave_id_uniform();
  const int wid = blockIdx.x * kWavesMixed + wave;
  const int t0 = __builtin_amdgcn_readfirstlane(first_tile(blockIdx.x, wave));
  const int t1 = __builtin_amdgcn_readfirstlane(first_tile(blockIdx.x, wave + 1));   // k = 4: s_off[b + 1]
  if (t1 <= t0) {
    if ((tid & (kWave - 1)) == 0) da.ws_cut[2 * wid] = -1;   // no tiles: nothing for the merge
    return;
  }
  dm::decode_worker<G>(da, s_pre, chunk, nch, wid, t0, t1 - t0, 0, 0);   // (uneven shares: the merge finds the last worker)
}

template <int G>
hipError_t launch_mixed_group(PrefillArgs pa, DecodeArgs da, MixedModel mm, int grid, hipStream_t stream) {
  da.num_workers = grid * kWavesMixed;
  // (block, KV head) rows of 4 KiB: 32-bit offsets reach them all below 2^20 rows
  if ((int64_t)pa.num_blocks * pa.num_kv_heads <= (int64_t)1 << 20)
    hipLaunchKernelGGL((mixed_kernel<G, true>), dim3(grid), dim3(kThreadsMixed), 0, stream, pa, da, mm);
  else
    hipLaunchKernelGGL((mixed_kernel<G, false>), dim3(grid), dim3(kThreadsMixed), 0, stream, pa, da, mm);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_decode_merge(da, G, stream);
}

}  // namespace

hipError_t launch_mixed(PrefillArgs pa, DecodeArgs da, MixedModel mm, int group, int num_units, hipStream_t stream) {
  // two workgroups per compute unit of the stream, as both halves run
  const int cus = stream_compute_units(stream);
  const int grid = 2 * cus;
  if (grid > 1024 || num_units > grid || pa.num_seqs * pa.tiles_per_seq > pf::kMaxRankItems)
    return hipErrorInvalidValue;
  pa.num_cus = 0;   // no splitting: a unit per workgroup
  pa.ws_o = nullptr;
  pa.ws_ml = nullptr;
  pa.ws_list = nullptr;
  pa.ws_slots = 0;
  pa.xcd_cus = (cus == stream_compute_units(nullptr) && cus % pf::kXcds == 0) ? cus / pf::kXcds : 0;
  switch (group) {
    case 1: return launch_mixed_group<1>(pa, da, mm, grid, stream);
    case 2: return launch_mixed_group<2>(pa, da, mm, grid, stream);
    case 4: return launch_mixed_group<4>(pa, da, mm, grid, stream);
    case 8: return launch_mixed_group<8>(pa, da, mm, grid, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace bros
