// Device code of the matrix-core prefill, shared by the prefill launch
// (prefill.hip) and the fused prefill|decode launch (mixed.hip).
// bros_attn_prefill_chunk (bf16) on gfx950 matrix cores.
//
// What it computes (Sec. 6: prefill rows of the mixed batch concatenated with a
// length table; chunked prefill on top of cached context, Sec. 2.2): row j of
// sequence s sits at position c0 + j, c0 = ctx - n, and attends to positions
// 0 .. c0 + j of the sequence, gathered from the bidirectional pool (Sec. 5.1).
//
// Work units. A workgroup (4 waves, one per SIMD) owns one (sequence, KV
// head, tile of 128 / G positions): 128 query rows, all G = Hq / Hkv query
// heads of that KV head. Waves 0-3 take rows 0-31, 32-63, 64-95, 96-127 over
// all the key tiles of the context. Two workgroups share a compute unit (77
// KiB of LDS each, two waves per SIMD), and they run unsynchronised: one
// wave's vector work (the softmax) runs beside the other's matrix-core
// products -- a single wave issues vector instructions at about half the rate
// two waves reach -- and one unit's start-up (lengths, Q, first tiles) hides
// behind the other's steps.
//
// Balance. All units of a step usually run in one round, so the kernel lasts
// as long as its longest unit. When the units are fewer than the compute
// units (a long context under few chunk rows) and a workspace is given, a
// unit whose key tiles exceed the part size T is split into ceil(tiles / T)
// pieces over disjoint key ranges, T = ceil(all tiles x Hkv / compute units)
// (at least kMinPartTiles). A split unit's pieces write unnormalised partial
// rows with their max and sum; prefill_merge_kernel folds them (the same
// max-rescaled sum as the decode's merge). Unsplit units write their rows
// directly. Units (or pieces) are launched longest first, ranked on the device
// from the length table, and consecutive ids are spread over the XCDs so that
// one KV head of every sequence stays on one XCD's L2.
//
// Data path. K and V rows go straight from the pool into LDS
// (global_load_lds, no registers), row-major [key][d] with the 16-byte chunks
// of row r permuted by chunk ^ swz(r), which makes both the K operand reads
// and the transposing V^T reads (ds_read_b64_tr_b16) free of bank conflicts
// (64 banks of 4 bytes).
// K and V have rings of their own (four slots each): the K tile of step i + 1
// is read while the V tile of step i is, and each slot is refilled four steps
// ahead of its use. The piece's table entries are validated once into LDS as
// (block, KV head) row indices, so a load's address is the row times 4 KiB
// plus the lane's offset (one vector add; below 2^20 rows the pool's rows all
// lie within 32-bit offsets of its base), and a tile's K and V loads, one
// step apart, share one index.
//
// The instruction stream of a step is what bounds it (a lone wave issues an
// instruction every 9 cycles or so), so the step carries as few as it can:
// no 64-bit address arithmetic, the row sums of P as two more matrix-core
// products (a ones operand times P^T) instead of eight dependent dot
// products, and the rescale factor computed only when the max moves.
//
// Software pipeline (per wave, per step): the scores S^T = K Q^T of the next
// tile are computed on the matrix cores while the vector ALU turns the current
// tile's scores into probabilities, then O^T += V^T P^T; the max of the next
// tile's scores decides the rescale before the step ends. In the transposed
// orientation lane l owns query row l % 32, so the row max needs one
// exchange between the two half-waves, the O rescale is lane-local, and the P
// operand is built straight from the score accumulators (keys are permuted
// identically in P and V^T; the sums over keys do not care). The causal
// mask compares each key's logical position with the row's position, only on
// tiles that reach the diagonal, the context end or an invalid table entry:
// direction only reorders keys inside a block, which neither product sees.
// V rows of slots that are not context are zeroed in LDS, so the matrix
// cores never multiply whatever the pool holds there. The running max moves
// lazily (only when a score exceeds it by more than 2^8), so the O rescale
// is rare.

#pragma once

#include "bros_device.h"
#include "bros_kernels.h"

#include <limits.h>
#include <math.h>

#include <type_traits>

namespace bros {
namespace pf {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2_t;
typedef __attribute__((__vector_size__(2 * sizeof(float)))) float float2_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float floatx16;
typedef unsigned v4u_t __attribute__((ext_vector_type(4)));
typedef short v4s_t __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;                      // 4 waves: one per SIMD, two workgroups per CU
constexpr int kRows = 128;                         // query rows per workgroup
constexpr int kKeys = 32;                          // keys per tile (2 blocks)
constexpr int kSlots = 4;                          // stages of the K ring and of the V ring
constexpr int kRowBytes = kHeadDim * 2;            // bytes of one K or V row
constexpr int kTileBytes = kKeys * kRowBytes;      // one K or V tile in LDS
constexpr float kRescaleSlack = 8.0f;              // log2 units
constexpr float kNoMax = -1.0e30f;
constexpr int kMaxTableLds = kPrefillMaxCtxMfma / kBlockSize;   // table entries staged in LDS
constexpr int kTablePad = 32;                      // staged entries past the last tile (loads run ahead)
constexpr int kMaxRankItems = kThreads;            // units planned on the device (one per thread)
constexpr int kMaxPieces = 2 * kThreads;           // pieces ranked on the device (two per thread)
constexpr int kMinPartTiles = 8;                   // the shortest piece a unit is split into
constexpr int kLoadsPerStep = 4;                   // two K and two V loads per wave per step
constexpr int kXcds = 8;                           // accelerator dies of the chip; blockIdx % 8 picks the die

__device__ __forceinline__ bf16x8_t as_bf16x8(v4u_t v) { return __builtin_bit_cast(bf16x8_t, v); }
__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {   // round to nearest even
  const float2_t f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}
// 16-byte chunk c of row r of a K or V tile sits at byte r * 256 + 16 * (c ^ swz(r)).
// The row's four bits are permuted (r1 r0 r2 r3): the 16 rows a K read
// serves in one pass see 16 different chunks, and the four keys a transposing
// V read serves in one pass (rows 4h .. 4h + 3, plus 8) see four different
// 64-byte groups, so neither read meets a bank conflict with 64 banks.
__device__ __forceinline__ int swz(int r) { return ((r & 3) << 2) | (((r >> 2) & 1) << 1) | ((r >> 3) & 1); }

__device__ __forceinline__ uint2 lds_read_tr(const uint8_t* p) {   // ds_read_b64_tr_b16
  const v4s_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (v4s_t __attribute__((address_space(3)))*)(p));
  return __builtin_bit_cast(uint2, v);
}
// 16 bytes per lane from `src` straight into LDS at dst + 16 * lane
// (global_load_lds_dwordx4; dst is wave-uniform, passed in M0). Issued as
// inline assembly so the compiler's own wait insertion neither sees these
// writes to LDS nor orders LDS reads of other ring slots behind them: the
// kernel's explicit waits (wait_vmem) and barriers order every access.
// The source is a wave-uniform base (scalar registers) plus a per-lane byte
// offset.
__device__ __forceinline__ void load_to_lds(const void* base, uint32_t lane_off, const uint8_t* dst) {
  // the LDS aperture is 4 GiB aligned: the low half of a generic pointer into
  // LDS is the LDS address
  const uint32_t m0 = (uint32_t)(uintptr_t)dst;
  asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(lane_off), "s"(base), "{m0}"(__builtin_amdgcn_readfirstlane(m0)));
}
// A load the compiler may issue as a scalar (uniform) load.
typedef const int32_t __attribute__((address_space(4)))* scalar_i32_ptr;
__device__ __forceinline__ int32_t load_uniform(const int32_t* p, size_t i) {
  return ((scalar_i32_ptr)p)[i];   // address-space cast: C-style only
}
// Workgroup barrier for the tile pipeline: this wave's LDS reads and writes
// are complete (lgkmcnt 0) and the compiler may not move memory accesses
// across it. Loads into LDS still in flight are not waited for here; each
// wave waits for its own loads (wait_vmem) before the barrier that publishes
// them.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}
// Wait until at most N of this wave's vector-memory operations are
// outstanding (they complete in order); a compiler barrier for memory.
template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// Maximum of x over lanes l and l ^ 32 (v_permlane32_swap).
__device__ __forceinline__ float pair_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int N>
using Int = std::integral_constant<int, N>;

// Key tiles of unit (s, t): the keys its last row sees, in tiles of kKeys; 0
// for a tile past the sequence's rows or inconsistent lengths.
// The same from the sequence's lengths: first row q_begin, n rows, context ctx_s.
__device__ __forceinline__ int unit_tiles_of(const PrefillArgs& a, int q_begin, int n, int ctx_s, int t, int qt) {
  const int t0 = t * qt;
  if (q_begin < 0 || n <= 0 || q_begin + n > a.num_q_tokens || t0 >= n) return 0;
  const int c0 = ctx_s - n;
  if (c0 < 0) return 0;
  const int ctx = min(ctx_s, min(a.max_ctx, a.max_blocks_per_seq * kBlockSize));
  const int kend = min(ctx, c0 + min(n, t0 + qt));
  return (kend + kKeys - 1) / kKeys;
}
__device__ __forceinline__ int unit_tiles(const PrefillArgs& a, int s, int t, int qt) {
  const int q_begin = a.cu_q[s];
  return unit_tiles_of(a, q_begin, a.cu_q[s + 1] - q_begin, a.ctx_lens[s], t, qt);
}

// Inclusive prefix sum of v over the workgroup's threads (thread order);
// *total gets the sum. `scratch` holds kThreads / kWave ints. Every thread
// of the workgroup calls it.
static __device__ int block_scan(int v, int* scratch, int* total) {
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int u = __shfl_up(v, o);
    if (lane >= o) v += u;
  }
  if (lane == kWave - 1) scratch[w] = v;
  __syncthreads();
  int before = 0, sum = 0;
#pragma unroll
  for (int i = 0; i < kThreads / kWave; ++i) {
    const int x = scratch[i];
    before += i < w ? x : 0;
    sum += x;
  }
  __syncthreads();
  *total = sum;
  return v + before;
}

// Index of the entry of rank `rank` among len[0 .. n), longest first (ties
// by index), or -1 past the last. len is 16-byte aligned LDS, padded with -1
// up to a multiple of 4 entries; s_res is one int of LDS. Every thread of the
// workgroup calls it; the result is uniform.
static __device__ int find_rank(const int* len, int n, int rank, int* s_res) {
  const int tid = threadIdx.x;
  if (tid == 0) *s_res = -1;
  __syncthreads();
  const int n4 = (n + 3) / 4;
  for (int k = tid; k < n; k += kThreads) {
    const int my = len[k];
    int r = 0;
    int j4 = 0;
    for (; j4 + 4 <= n4; j4 += 4) {   // four reads in flight
      int4 l4[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) l4[u] = reinterpret_cast<const int4*>(len)[j4 + u];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int lj[4] = {l4[u].x, l4[u].y, l4[u].z, l4[u].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) r += (lj[e] > my) | ((lj[e] == my) & (4 * (j4 + u) + e < k));
      }
    }
    for (; j4 < n4; ++j4) {
      const int4 l4 = reinterpret_cast<const int4*>(len)[j4];
      const int lj[4] = {l4.x, l4.y, l4.z, l4.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) r += (lj[e] > my) | ((lj[e] == my) & (4 * j4 + e < k));
    }
    if (r == rank) *s_res = k;
  }
  __syncthreads();
  return __builtin_amdgcn_readfirstlane(*s_res);
}

// What a workgroup of the prefill grid works on: key tiles
// [part L / parts, (part + 1) L / parts) of unit (item, KV head), L being the
// unit's key tiles. Split units (parts > 1) keep their partial rows in
// workspace slots first_slot .. first_slot + parts - 1 (times Hkv).
struct PiecePlan {
  int item;         // -1: nothing for this rank
  int part;
  int parts;
  int first_slot;
  int q_begin, n, ctx;   // the item's sequence: cu_q[s], cu_q[s + 1] - cu_q[s], ctx_lens[s] (n = -1: not read)
};

// The piece of rank `rank` (longest first). Items are (sequence, tile of
// positions); all KV heads of an item have its length L (key tiles of its
// last row). Without splitting (num_cus 0) each item is one piece. With it,
// the part size is T = max(kMinPartTiles, ceil(sum L x Hkv / num_cus)), the
// mean work of a compute unit, and an item becomes ceil(L / T) pieces; then
// ranks exceed the items by at most num_cus / Hkv and split pieces times Hkv
// number at most 2 num_cus. Workgroup 0 writes the list of split items for
// the merge. `scratch` is 2 kMaxPieces + 4 + kThreads / kWave + 3
// kMaxRankItems ints of LDS, 16-byte aligned, that nothing else uses
// meanwhile. Every thread of the workgroup calls it. The lengths read for the
// ranking come back with the plan, so the unit does not read them again.
template <int QT>
__device__ PiecePlan plan_pieces(const PrefillArgs& a, int rank, int* scratch) {
  const int tid = threadIdx.x;
  const int tps = a.tiles_per_seq;
  const int n_items = a.num_seqs * tps;
  if (n_items > kMaxRankItems) {
    // (never split) the longest tile of every sequence first
    const int t_rank = rank / a.num_seqs;
    return PiecePlan{t_rank < tps ? (rank % a.num_seqs) * tps + (tps - 1 - t_rank) : -1, 0, 1, 0, 0, -1, 0};
  }
  int* s_len = scratch;                     // [kMaxPieces] lengths, then -1 padding
  int* s_pid = scratch + kMaxPieces;        // [kMaxPieces] item * 1024 + part
  int* s_res = scratch + 2 * kMaxPieces;    // [4]
  int* s_red = s_res + 4;                   // [kThreads / kWave]
  int* s_seq = s_red + kThreads / kWave;    // [3 kMaxRankItems] per item: q_begin, n, ctx
  int L = -1;
  if (tid < n_items) {
    const int sq = tid / tps;
    const int q0 = a.cu_q[sq], q1 = a.cu_q[sq + 1], cx = a.ctx_lens[sq];
    L = unit_tiles_of(a, q0, q1 - q0, cx, tid % tps, QT);
    s_seq[3 * tid] = q0;
    s_seq[3 * tid + 1] = q1 - q0;
    s_seq[3 * tid + 2] = cx;
  }
  auto lens_of = [&](PiecePlan p) -> PiecePlan {   // (the item's entries were written before a barrier)
    if (p.item >= 0) {
      p.q_begin = s_seq[3 * p.item];
      p.n = s_seq[3 * p.item + 1];
      p.ctx = s_seq[3 * p.item + 2];
    }
    return p;
  };
  int P = 1, n_pieces = n_items, pbase = tid, sbase = 0;
  bool split = false;
  if (a.num_cus > 0) {
    int total = 0;
    block_scan(max(L, 0), s_red, &total);
    const int T = max(kMinPartTiles, (int)(((int64_t)total * a.num_kv_heads + a.num_cus - 1) / a.num_cus));
    const int Pt = L > 0 ? 1 + (L - 1) / T : 0;
    const int pend = block_scan(Pt, s_red, &n_pieces);
    const int own = Pt > 1 ? Pt : 0;
    int n_split = 0;
    const int send = block_scan(own, s_red, &n_split);
    split = n_split > 0 && n_pieces <= kMaxPieces && (int64_t)n_split * a.num_kv_heads <= a.ws_slots;
    if (split) {
      P = Pt;
      pbase = pend - Pt;
      sbase = send - own;
    } else {
      n_pieces = n_items;
    }
    if (blockIdx.x == 0) {
      // the split items, in item order: count, then (item, parts, first slot)
      int count = 0;
      const int is = split && P > 1 ? 1 : 0;
      const int idx = block_scan(is, s_red, &count) - is;
      if (is) {
        a.ws_list[1 + 3 * idx] = tid;
        a.ws_list[2 + 3 * idx] = P;
        a.ws_list[3 + 3 * idx] = sbase;
      }
      if (tid == 0) a.ws_list[0] = split ? count : 0;
    }
  }
  if (!split) {
    if (tid < kMaxRankItems) s_len[tid] = L;   // -1 past the items
    const int k = find_rank(s_len, n_items, rank, s_res);
    const PiecePlan out = lens_of(PiecePlan{k, 0, 1, 0, 0, -1, 0});
    __syncthreads();   // the scratch is the caller's again
    return out;
  }
  if (tid < n_items) {
    for (int q = 0; q < P; ++q) {
      s_len[pbase + q] = (int)((int64_t)(q + 1) * L / P) - (int)((int64_t)q * L / P);
      s_pid[pbase + q] = tid * 1024 + q;
    }
  }
  if (tid < ((n_pieces + 3) & ~3) - n_pieces) s_len[n_pieces + tid] = -1;   // padding
  const int k = find_rank(s_len, n_pieces, rank, s_res);
  PiecePlan out{-1, 0, 0, 0, 0, -1, 0};
  if (k >= 0) {
    const int id = s_pid[k];
    const int item = id / 1024;
    if (tid == item) {
      s_res[1] = P;
      s_res[2] = sbase;
    }
    __syncthreads();
    out = lens_of(PiecePlan{item, id % 1024, s_res[1], s_res[2], 0, -1, 0});
  }
  __syncthreads();   // the scratch is the caller's again
  return out;
}

// Workgroup b of a first round that has the whole chip, as a unit id. Ids
// r * Hkv + g give every rank all KV heads on consecutive ids, i.e. on
// different XCDs (id % 8), and one KV head of every unit on one XCD when Hkv
// is a multiple of 8. Workgroup j of an XCD (blockIdx = 8 j + x) first lands
// on compute unit j of the XCD, and workgroup j + C (C compute units per XCD)
// on the same unit's second slot; the second slots take the remaining ranks
// in reverse, so the longest unit of a compute unit shares it with the
// shortest and every unit's pair carries about the same work.
__device__ __forceinline__ int paired_id(const PrefillArgs& a, int b, int grid) {
  int id = b;
  if (a.xcd_cus > 0) {
    const int x = id % kXcds, j = id / kXcds;
    const int C = a.xcd_cus;
    const int R = min((grid - x + kXcds - 1) / kXcds, 2 * C);   // this XCD's first-round workgroups
    if (j >= C && j < R) id = (R - 1 - (j - C)) * kXcds + x;
  }
  return id;
}

// LDS of one unit: the K ring and the V ring, kSlots slots of one 32-key tile
// each (1024-byte aligned), and the sequence's validated table entries and
// directions. Declared by each kernel, so that slot offsets stay compile-time
// constants that fold into the LDS instructions' offset field.
#define BROS_PREFILL_UNIT_LDS                                                                   \
  __shared__ __attribute__((aligned(1024))) uint8_t s_kring[::bros::pf::kSlots * ::bros::pf::kTileBytes]; \
  __shared__ __attribute__((aligned(1024))) uint8_t s_vring[::bros::pf::kSlots * ::bros::pf::kTileBytes]; \
  __shared__ int s_first_bad;                                                                   \
  __shared__ int s_tbl[::bros::pf::kMaxTableLds + ::bros::pf::kTablePad];                      \
  __shared__ int8_t s_dir[::bros::pf::kMaxTableLds + ::bros::pf::kTablePad];

// One unit (or piece) of the matrix-core prefill: unit id `id` (rank id /
// Hkv, KV head id % Hkv), run by the calling workgroup's four waves. Every
// early return is uniform over the workgroup.
template <int G, bool kOff32>
__device__ __forceinline__ void prefill_unit(const PrefillArgs& a, int id, uint8_t* s_kring, uint8_t* s_vring,
                                             int* s_first_bad_p, int* s_tbl, int8_t* s_dir) {
  constexpr int QT = kRows / G;   // positions per unit
  constexpr int kSlotBytes = kTileBytes;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wv = wave_id_uniform();
  const int rg = wv & 3;    // row group: rows 32 rg .. 32 rg + 31

  const int Hkv = a.num_kv_heads;
  const int tps = a.tiles_per_seq;
  const int g = id % Hkv;
  const int rank = id / Hkv;
  // (the K ring is free until the first loads)
  const PiecePlan plan = plan_pieces<QT>(a, rank, reinterpret_cast<int*>(s_kring));
  const int item = __builtin_amdgcn_readfirstlane(plan.item);
  if (item < 0) return;                      // a rank past the last piece
  const int part = __builtin_amdgcn_readfirstlane(plan.part);
  const int parts = __builtin_amdgcn_readfirstlane(plan.parts);
  const int pslot = __builtin_amdgcn_readfirstlane(plan.first_slot);
  const int s = item / tps;
  const int t = item % tps;

  // The unit's lengths: from the ranking, else as scalar loads.
  int q_begin, n, ctx_s;
  if (__builtin_amdgcn_readfirstlane(plan.n) >= 0) {
    q_begin = __builtin_amdgcn_readfirstlane(plan.q_begin);
    n = __builtin_amdgcn_readfirstlane(plan.n);
    ctx_s = __builtin_amdgcn_readfirstlane(plan.ctx);
  } else {
    q_begin = load_uniform(a.cu_q, s);
    n = load_uniform(a.cu_q, s + 1) - q_begin;
    ctx_s = load_uniform(a.ctx_lens, s);
  }
  const int t0 = t * QT;
  if (q_begin < 0 || n <= 0 || q_begin + n > a.num_q_tokens || t0 >= n || ctx_s < n) return;
  const int c0 = ctx_s - n;
  const int ctx = min(ctx_s, min(a.max_ctx, a.max_blocks_per_seq * kBlockSize));
  const int kend = min(ctx, c0 + min(n, t0 + QT));
  const int unit_kt = (kend + kKeys - 1) / kKeys;   // key tiles of the unit
  // this piece's key tiles [kb, kb + n_kt)
  const int kb = (int)((int64_t)part * unit_kt / parts);
  const int n_kt = (int)((int64_t)(part + 1) * unit_kt / parts) - kb;
  if (n_kt <= 0) return;
  const int nblk = (ctx + kBlockSize - 1) / kBlockSize;
  // keys below this logical position are visible to every row of the unit
  const int full_below = min(ctx, c0 + t0 + 1);

  const int half = lane >> 5;
  const int mrow = lane & 31;
  const int Hq = a.num_q_heads;
  const int r_unit = 32 * rg + mrow;            // the lane's row in the unit
  const int head = g * G + r_unit / QT;
  const int qrow = t0 + r_unit % QT;
  const bool row_valid = qrow < n;
  const int qpos = row_valid ? c0 + qrow : -1;
  const size_t row_off = ((size_t)(q_begin + min(qrow, n - 1)) * Hq + head) * kHeadDim;   // q / out row

  // Q^T operand: for d-step c, lane holds Q[row][16c + 8*half .. +8). Issued
  // before every load into LDS, so waiting for the first tiles covers it.
  bf16x8_t qf[8];
  {
    const uint16_t* qp = static_cast<const uint16_t*>(a.q) + row_off;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      v4u_t v = {0, 0, 0, 0};
      if (row_valid) v = *reinterpret_cast<const v4u_t*>(qp + 16 * c + 8 * half);
      qf[c] = as_bf16x8(v);
    }
  }

  // Table entries. The first few come in as scalar loads; the piece's
  // entries are then staged in LDS as (block, KV head) row indices,
  // b * Hkv + g, with direction flags (0 for an entry that is invalid, past
  // the context or outside the piece, whose index is 0: a load from there
  // fills a slot nobody reads, so every step issues exactly kLoadsPerStep
  // loads and the waits below can count). The tile of step j is kb + j; this
  // wave loads, positions and fixes up rows 8 rg .. 8 rg + 7 of it, in block
  // rg / 2.
  const uint16_t* kpool = static_cast<const uint16_t*>(a.k_pool);
  const uint16_t* vpool = static_cast<const uint16_t*>(a.v_pool);
  const int32_t* tbl = a.block_tables + (size_t)s * a.max_blocks_per_seq;
  const int blo = 2 * kb, bhi = min(nblk, 2 * (kb + n_kt));   // the piece's entries
  auto entry = [&](int b) -> int {
    const int v = load_uniform(tbl, min(max(b, 0), nblk - 1));
    return (b >= blo && b < bhi && v >= 0 && v < a.num_blocks) ? v * Hkv + g : 0;
  };
  const int my_bt = rg >> 1;                // block of the tile holding this wave's rows
  const int my_slot0 = 8 * (rg & 1);        // first of its slots
  // This wave's row index for step j (a vector register holding a uniform value).
  auto own = [&](int j) -> int { return s_tbl[2 * (kb + j) + my_bt]; };

  // Loads: load i (0, 1) covers tile rows 8 rg + 4i + lane / 16, lane writing
  // physical chunk lane % 16, which holds logical chunk (lane % 16) ^ swz(row).
  const int ld_slot = lane >> 4;
  uint32_t ld_off[2];   // byte offset of the lane's 16 bytes within the block
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int row = 8 * rg + 4 * i + ld_slot;   // tile row
    ld_off[i] = (uint32_t)(((my_slot0 + 4 * i + ld_slot) * kHeadDim + (((lane & 15) ^ swz(row)) << 3)) * 2);
  }
  // A (block, head) row is 4 KiB. With kOff32 the pool's rows all lie within
  // 4 GiB of its base, so the per-lane offset carries the row (one vector add
  // per load); else the base moves by the row, in scalar registers.
  auto issue = [&](int idx, const uint16_t* pool, uint8_t* ring) __attribute__((always_inline)) {
    uint8_t* dst = ring + 8 * rg * kRowBytes;
    if constexpr (kOff32) {
#pragma unroll
      for (int i = 0; i < 2; ++i) load_to_lds(pool, ld_off[i] + ((uint32_t)idx << 12), dst + 4 * i * kRowBytes);
    } else {
      const uint16_t* base = pool + (size_t)__builtin_amdgcn_readfirstlane(idx) * (kBlockSize * kHeadDim);
#pragma unroll
      for (int i = 0; i < 2; ++i) load_to_lds(base, ld_off[i], dst + 4 * i * kRowBytes);
    }
  };
  // Once this wave's V loads of step j have landed: zero its rows whose slot
  // is not context.
  auto fixup_v = [&](int j, uint8_t* ring) __attribute__((always_inline)) {
    if (j >= n_kt) return;
    const int b = 2 * (kb + j) + my_bt;
    const int dirv = __builtin_amdgcn_readfirstlane((int)s_dir[b]);
    if (dirv != 0 && (b + 1) * kBlockSize <= ctx) return;
    uint8_t* dv = ring + 8 * rg * kRowBytes;
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int r8 = 4 * p + ld_slot;   // row among the wave's 8
      if (!(dirv != 0 && b * kBlockSize + slot_of_offset(my_slot0 + r8, dirv) < ctx))
        *reinterpret_cast<v4u_t*>(dv + r8 * kRowBytes + (lane & 15) * 16) = v4u_t{0, 0, 0, 0};
    }
  };

  // K operand (S^T = K Q^T, d-step c): tile row mrow, logical chunk 2c + half.
  const int k_sw = swz(mrow);
  const int k_lane = mrow * kRowBytes + (((half ^ k_sw) & 1) << 4);
  // V^T operand via the transposing read, per (dt, part): lane (group j = lane /
  // 16, q = lane % 4, t = lane % 16 / 4) reads dims 32dt + 16(j % 2) + 4q ..+3 of
  // key 16c2 + 8part + 4half + t (key order shared with the P operand).
  const int tr_j = lane >> 4, tr_q = lane & 3, tr_t = (lane >> 2) & 3;
  int v_off[2];
  int v_sw[2];
#pragma unroll
  for (int part = 0; part < 2; ++part) {
    const int key = 8 * part + 4 * half + tr_t;
    v_sw[part] = swz(key);
    v_off[part] = key * kRowBytes + ((((2 * (tr_j & 1) + (tr_q >> 1)) ^ v_sw[part]) & 3) << 4) + (tr_q & 1) * 8;
  }

  floatx16 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o[dt] = floatx16{};
  float m_run = kNoMax, m_prev = kNoMax;
  // Row sums of P on the matrix cores: a ones operand times P^T gives, in
  // every accumulator of lane l, the sum over the tile's keys of row l % 32
  // (both half-waves get the whole sum). Only element 0 is read (and
  // rescaled); the others accumulate along unread.
  floatx16 lacc = floatx16{};
  const bf16x2_t one2 = {(__bf16)1.0f, (__bf16)1.0f};
  const v4u_t ones4 = {__builtin_bit_cast(uint32_t, one2), __builtin_bit_cast(uint32_t, one2),
                       __builtin_bit_cast(uint32_t, one2), __builtin_bit_cast(uint32_t, one2)};
  // Raw scores of the wave's next tile, carried from the step that computes
  // them (and their max) to the step that turns them into probabilities: two
  // buffers, so that a step reads one while the matrix cores write the other
  // (the unrolled main loop alternates them; elsewhere `sa` is the carried one).
  // Every accumulator here lives in vector registers: with no accumulation
  // register in use, the compiler gives the wave its whole register budget as
  // vector registers and the matrix cores write their results there, so the
  // vector ALU reads scores and rescales O directly.
  floatx16 sa, sb;
  const float sl2 = a.scale_log2;

  // K operands of the tile in K ring `sk`, all eight d-steps, issued
  // together.
  auto k_operands = [&](const uint8_t* sk, v4u_t (&kv)[8]) __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < 8; ++c) kv[c] = *reinterpret_cast<const v4u_t*>(sk + k_lane + (((2 * c) ^ (k_sw & 14)) << 4));
  };
  // S^T = K Q^T (one dependent chain; back-to-back accumulation needs no gap).
  auto scores = [&](const v4u_t (&kv)[8], floatx16& acc) __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < 8; ++c)
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kv[c]), qf[c], c == 0 ? floatx16{} : acc, 0, 0, 0);
  };
  // Mask the accumulators in place (when asked: `tile` is the tile they
  // belong to) and fold the tile's max into the running max; sets alpha, the
  // factor O and l take for the new max. Accumulator j is key
  // k = 8*(j/4) + 4*half + j%4 of the tile: physical slot k % 16 of the
  // tile's block k / 16, which holds that block's position offset
  // slot_of_offset(k % 16, dir).
  auto mask_max = [&](floatx16& cur, auto maskc, int tile) __attribute__((always_inline)) {
    if constexpr (decltype(maskc)::value) {
      // visible: valid block, position < ctx and <= the row's position
      const int lim = min(qpos, ctx - 1);
      const int dir0 = s_dir[2 * tile];       // 0: invalid, past the context or outside the piece
      const int dir1 = s_dir[2 * tile + 1];
      const bool ok0 = dir0 != 0, ok1 = dir1 != 0;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int k = 8 * (j >> 2) + 4 * half + (j & 3);   // j is a constant; half per lane
        const int pos = 32 * tile + (k & 16) + slot_of_offset(k & 15, (j >> 3) ? dir1 : dir0);
        const bool ok = (j >> 3) ? ok1 : ok0;   // k / 16 == j / 8
        cur[j] = (ok && pos <= lim) ? cur[j] : -INFINITY;
      }
    }
    float mr = -INFINITY;   // max of the raw scores (the scale > 0 commutes with max)
#pragma unroll
    for (int j = 0; j < 16; ++j) mr = fmaxf(mr, cur[j]);
    const float mx = pair_max(mr) * sl2;   // log2 units; -inf when nothing is visible
    m_prev = m_run;
    m_run = mx > m_run + kRescaleSlack ? mx : m_run;
  };
  // P = exp2(S * scale - m) rounded to bf16 (the P^T operands); the row sums
  // (lacc) add exactly these rounded weights, the ones the PV product
  // applies. Operand c2 (16 keys) holds accumulators 8*c2 .. 8*c2 + 7.
  auto probs = [&](bf16x8_t (&pf)[2], const floatx16& cur) __attribute__((always_inline)) {
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2) {
      bf16x2_t pw[4];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float2_t pp = {fast_exp2(fmaf(cur[8 * c2 + 2 * w], sl2, -m_run)),
                             fast_exp2(fmaf(cur[8 * c2 + 2 * w + 1], sl2, -m_run))};
        pw[w] = __builtin_convertvector(pp, bf16x2_t);   // round to nearest even
      }
      const v4u_t pk = {__builtin_bit_cast(uint32_t, pw[0]), __builtin_bit_cast(uint32_t, pw[1]),
                        __builtin_bit_cast(uint32_t, pw[2]), __builtin_bit_cast(uint32_t, pw[3])};
      pf[c2] = as_bf16x8(pk);
    }
  };
  // V^T operands of the tile in V ring `sv` for key step c2.
  auto v_operands = [&](const uint8_t* sv, int c2, v4u_t (&vv)[4]) __attribute__((always_inline)) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      // chunk 4dt + (2(j % 2) + q / 2) of the row: the dt bits XOR the swizzle's high bits
      const uint2 lo = lds_read_tr(sv + 16 * c2 * kRowBytes + v_off[0] + (((4 * dt) ^ (v_sw[0] & 12)) << 4));
      const uint2 hi = lds_read_tr(sv + 16 * c2 * kRowBytes + v_off[1] + (((4 * dt) ^ (v_sw[1] & 12)) << 4));
      vv[dt] = v4u_t{lo.x, lo.y, hi.x, hi.y};
    }
  };
  // O^T += V^T P^T for key step c2.
  auto pv = [&](const v4u_t (&vv)[4], const bf16x8_t (&pf)[2], int c2) __attribute__((always_inline)) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
      o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vv[dt]), pf[c2], o[dt], 0, 0, 0);
    lacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(ones4), pf[c2], lacc, 0, 0, 0);
  };
  // Rare (lazy max).
  auto rescale_o = [&]() __attribute__((always_inline)) {
    if (__builtin_amdgcn_ballot_w64(m_run != m_prev) != 0) {
      const float alpha = fast_exp2(m_prev - m_run);
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) o[dt] *= alpha;
      lacc[0] *= alpha;
    }
  };

  // One step of this wave: P and PV for its current tile (V in `sv`) and, when
  // it has a next tile, that tile's scores (K in `sk`), mask (for tile
  // `next_tile`) and max. In program order the LDS reads go first; then the
  // next tile's score products, which the matrix cores run while the vector
  // ALU forms the current probabilities; then the PV products, while the new
  // scores are masked and maxed. The compiler interleaves the phases freely
  // (scheduling barriers between them measured 1.5-4 % slower); the other
  // wave on the SIMD fills the gaps.
  // `in` holds the current tile's scores, `out` receives the next tile's.
  auto step = [&](const uint8_t* sk, const uint8_t* sv, int next_tile, auto has_next, auto mask_next,
                  const floatx16& in, floatx16& out) __attribute__((always_inline)) {
    constexpr bool NEXT = decltype(has_next)::value;
    v4u_t kv[8];
    v4u_t vv0[4], vv1[4];
    if constexpr (NEXT) k_operands(sk, kv);
    v_operands(sv, 0, vv0);
    bf16x8_t pf[2];
    if constexpr (NEXT) scores(kv, out);
    probs(pf, in);
    v_operands(sv, 1, vv1);
    pv(vv0, pf, 0);
    pv(vv1, pf, 1);
    if constexpr (NEXT) mask_max(out, mask_next, next_tile);
  };
  // After step ii: wait for batch ii + 1 (K of step ii + 2, V of step ii + 1),
  // zero V's non-context rows (FIX; a tile below plain_tiles has none),
  // publish, then issue batch ii + 4 into the slots step ii freed (K slot
  // (ii + 1) % 4, V slot ii % 4): K of step ii + 5 from row index ik, V of
  // step ii + 4 from iv.
  auto advance = [&](int ii, int sl, int ik, int iv, auto fixc) __attribute__((always_inline)) {
    const int sl1 = (sl + 1) & (kSlots - 1);
    wait_vmem<2 * kLoadsPerStep>();
    if constexpr (decltype(fixc)::value) fixup_v(ii + 1, s_vring + sl1 * kSlotBytes);
    lds_barrier();
    issue(ik, kpool, s_kring + sl1 * kSlotBytes);
    issue(iv, vpool, s_vring + sl * kSlotBytes);
  };
  const uint8_t* kr = s_kring;
  const uint8_t* vr = s_vring;

  // ---- Prologue. Step j's K tile lives in K slot j % 4, its V tile in V
  // slot j % 4. Batch b = (K of step b + 1, V of step b) is issued after
  // step b - 4 frees both slots. K of step 0 and batch 0 go first, together
  // with Q; batches 1 .. 3 follow once the first scores are in. (The first
  // row indices come as scalar loads; the LDS copy is made while they load.)
  auto own0 = [&](int j) -> int { return entry(2 * (kb + j) + my_bt); };
  const int e0 = own0(0);
  const int w0 = own0(1), w1 = own0(2), w2 = own0(3), w3 = own0(4);
  issue(e0, kpool, s_kring);
  issue(w0, kpool, s_kring + 1 * kSlotBytes);
  issue(e0, vpool, s_vring);
  // Tiles below `plain_tiles` need no mask: every key is context, sits behind
  // a valid table entry and is visible to every row of the unit. The first
  // invalid entry of the piece comes from the staging pass, while the first
  // tiles are in flight. Entries past the piece (read by loads that run
  // ahead) are staged as row 0 with direction 0.
  if (tid == 0) (*s_first_bad_p) = bhi;
  __syncthreads();
  for (int b = blo + tid; b < 2 * (kb + n_kt) + kTablePad; b += kThreads) {
    int idx = 0, d = 0;
    if (b < bhi) {
      const int v = tbl[b];
      if (v >= 0 && v < a.num_blocks) {
        idx = v * Hkv + g;
        d = entry_direction(a.dir, a.cls, a.dir_per_entry, a.max_blocks_per_seq, s, b);
      } else {
        atomicMin(s_first_bad_p, b);
      }
    }
    s_tbl[b] = idx;
    s_dir[b] = (int8_t)d;
  }
  __syncthreads();
  const int first_bad = __builtin_amdgcn_readfirstlane((*s_first_bad_p));
  const int plain_tiles = min(full_below / kKeys, first_bad / 2);
  // Everything so far, Q included: a wait the compiler sees, so it knows the
  // Q registers are ready and adds no wait of its own later.
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
  fixup_v(0, s_vring);
  lds_barrier();
  {
    v4u_t kv[8];
    k_operands(kr, kv);
    scores(kv, sa);
    if (kb >= plain_tiles) mask_max(sa, std::true_type{}, kb);
    else mask_max(sa, std::false_type{}, kb);
  }
  lds_barrier();   // K slot 0 is free again
  issue(w1, kpool, s_kring + 2 * kSlotBytes);
  issue(w0, vpool, s_vring + 1 * kSlotBytes);
  issue(w2, kpool, s_kring + 3 * kSlotBytes);
  issue(w1, vpool, s_vring + 2 * kSlotBytes);
  issue(w3, kpool, s_kring);
  issue(w2, vpool, s_vring + 3 * kSlotBytes);

  // ---- Steps. Before step i: batch i (K of step i + 1, V of step i) is in
  // LDS, batches i + 1 .. i + 3 are in flight. The steady state (this wave has
  // a next tile and it needs no mask) runs unrolled by the ring size, with
  // the slots as constants; the rest (the tiles at the diagonal or the context
  // end, a tile behind an invalid table entry, the last tile) runs in
  // separate loops with the slot as a variable. A tile's K and V loads use
  // the same row index, one step apart: `iv` carries it from the K load to
  // the V load.
  int ii = 0;
  int iv = w3;
  // the piece's tiles below plain_tiles, as a step bound
  const int n_plain = max(0, min(n_kt, plain_tiles - kb));
  auto main_step = [&](auto uc) __attribute__((always_inline)) -> bool {
    constexpr int u = decltype(uc)::value;
    if (ii + 1 >= n_plain) return false;
    const int ik = own(ii + 5);
    // step ii reads buffer ii % 2 and fills the other (u and ii agree mod 4)
    if constexpr (u % 2 == 0)
      step(kr + ((u + 1) % kSlots) * kSlotBytes, vr + u * kSlotBytes, 0, std::true_type{}, std::false_type{}, sa, sb);
    else
      step(kr + ((u + 1) % kSlots) * kSlotBytes, vr + u * kSlotBytes, 0, std::true_type{}, std::false_type{}, sb, sa);
    rescale_o();
    advance(ii, u, ik, iv, std::false_type{});
    iv = ik;
    ++ii;
    return true;
  };
  while (main_step(Int<0>{}) && main_step(Int<1>{}) && main_step(Int<2>{}) && main_step(Int<3>{})) {
  }
  if (ii & 1) sa = sb;   // the rest carries the scores in `sa`
  // Tiles with a next tile that needs (or may need) the mask.
  for (; ii + 1 < n_kt; ++ii) {
    const int sl = ii & (kSlots - 1);
    const int sl1 = (sl + 1) & (kSlots - 1);
    const int ik = own(ii + 5);
    step(kr + sl1 * kSlotBytes, vr + sl * kSlotBytes, kb + ii + 1, std::true_type{}, std::true_type{}, sa, sb);
    sa = sb;
    rescale_o();
    advance(ii, sl, ik, iv, std::true_type{});
    iv = ik;
  }
  // The last tile (no next tile to score).
  if (ii < n_kt) {
    const int sl = ii & (kSlots - 1);
    const int ik = own(ii + 5);
    step(kr, vr + sl * kSlotBytes, 0, std::false_type{}, std::false_type{}, sa, sb);
    advance(ii, sl, ik, iv, std::true_type{});
    iv = ik;
    ++ii;
  }
  wait_vmem<0>();
  const float l_run = lacc[0];
  if (parts > 1) {
    // ---- A piece of a split unit: unnormalised rows plus their max and sum.
    const size_t slot = ((size_t)(pslot + part) * Hkv + g) * kRows + r_unit;
    float* po = a.ws_o + slot * kHeadDim;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        const int d0 = 32 * dt + 8 * jq + 4 * half;   // accumulators 4jq..4jq+3 are dims d0..d0+3
        *reinterpret_cast<float4*>(po + d0) =
            make_float4(o[dt][4 * jq], o[dt][4 * jq + 1], o[dt][4 * jq + 2], o[dt][4 * jq + 3]);
      }
    }
    if (half == 0) {
      a.ws_ml[2 * slot] = m_run;
      a.ws_ml[2 * slot + 1] = l_run;
    }
    return;
  }
  // ---- A whole unit: normalise and write the rows.
  const float inv = l_run > 0.0f ? 1.0f / l_run : 0.0f;
  if (row_valid) {
    uint16_t* op = static_cast<uint16_t*>(a.out) + row_off;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        const int d0 = 32 * dt + 8 * jq + 4 * half;   // accumulators 4jq..4jq+3 are dims d0..d0+3
        uint2 w;
        w.x = pack2_bf16(o[dt][4 * jq + 0] * inv, o[dt][4 * jq + 1] * inv);
        w.y = pack2_bf16(o[dt][4 * jq + 2] * inv, o[dt][4 * jq + 3] * inv);
        *reinterpret_cast<uint2*>(op + d0) = w;
      }
    }
  }
}

}  // namespace pf
}  // namespace bros
