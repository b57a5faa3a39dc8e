// bros_attn_decode (bf16) on gfx950: paged decode attention over the
// bidirectional pool on the matrix cores (fp32 runs on the vector ALU,
// decode_f32.hip).
//
// What it computes (Sec. 2.1 decode attention over the cached KV; Sec. 5.1
// bidirectional slot order; Sec. 6 direction-aware paged kernel): for query
// row r of sequence s and query head h in KV group g = h / G,
//     out[r][h] = sum_p softmax_p(scale * q[r][h] . K[p][g]) V[p][g],  p < ctx(r),
// with the softmax taken online (running max and sum, Sec. 8's online-softmax
// kernels) and partial results over disjoint parts of a context combined by
// max-rescaling.
//
// Work. A tile is one (row, KV head, 16-slot block); a (row, KV head) pair is
// a segment of consecutive tiles. The grid holds what the compute units of
// the stream keep resident at two waves per SIMD, and every wave is an
// independent worker that takes an equal contiguous share of all tiles in
// (row, KV head, block) order, so the load is balanced to within one tile
// whatever the mix of context lengths. A worker walks its share tile by tile
// with kDepth register sets for K and V: while it computes tile i, the loads
// of the next kDepth - 1 tiles are in flight, and tile i + kDepth's are
// requested into tile i's set as soon as those registers are read (a tile may
// start a new segment). Fewer waves with more tiles in flight each move more
// bytes than more waves with one tile each: two waves per SIMD with two tiles
// in flight beat four waves with one by 5-8 %, and a third tile adds nothing.
// Block-table entries come through the scalar cache one tile before their
// loads issue. KV tiles are read with non-temporal loads; each byte of the KV
// pool is read once.
//
// A segment that lies wholly inside one worker's share is normalised and
// written by that worker. A segment cut between workers leaves one partial
// (m, l, acc) per worker, stored at slot (segment + worker) -- unique, since
// worker ranges are ordered like segments -- and the merge kernel folds them.
//
// Direction only decides which physical slots hold valid positions: attention
// is a sum over the cached tokens, so each score is paired with the V row of
// the same physical slot, and the logical position b*16 + (dir > 0 ? slot :
// 15 - slot) is compared with the context length in the tail block. Invalid
// slots are removed by selection (scores -inf, V zeroed), never by
// multiplication, so a peer request's tokens or NaNs there cannot leak.
#include "decode_common.h"

#include <mutex>
#include <type_traits>

namespace bros {
namespace {

constexpr int kMaxSplitBlocks = 64;   // fp32 split-K: blocks per split at most
// Tiles whose K/V loads a bf16 decode wave keeps in flight (register sets).
constexpr int kDepth = 2;

// ---------------------------------------------------------------------------
// bf16 decode on the matrix cores. Per 16-slot block of one (row, KV head), the
// G query heads of the group form a dense 16 x G x 128 contraction:
//   S^T[slot][head] = K[slot][:] . q[head][:]     mfma 16x16x32 (N = heads, padded)
//   O^T[dim][head] += V^T[dim][slot] P^T[slot][head]   mfma 16x16x16
// Lane l = 16 grp + col. In the C layout of the first product lane l holds the
// scores of slots 4 grp .. 4 grp + 3 for head col, which is exactly the B layout
// the second product wants for P^T: the softmax weights never move between
// lanes. The contraction index of the first product is a permutation of the
// head dims (K and q use the same one), and row m of output tile t is dim
// 8 m + t, so every operand comes from plain 16-byte loads: K slot col, dims
// 32 c + 8 grp ..; V slots 4 grp + j, dims 8 col ..; and lane l ends up holding
// dims 32 grp .. 32 grp + 31 of head col. Lanes with col >= G compute padding
// that is never stored.
// ---------------------------------------------------------------------------
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef short short4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float floatx4_t;

__device__ __forceinline__ v4u_t load_nt(const void* base, size_t elem) {
  return __builtin_nontemporal_load(reinterpret_cast<const v4u_t*>(static_cast<const uint16_t*>(base) + elem));
}

typedef const int32_t __attribute__((address_space(4)))* scalar_i32_ptr;

// A wave-uniform int32 read through the scalar cache (read-only data only).
__device__ __forceinline__ int32_t load_uniform(const int32_t* p, size_t i) {
  return ((scalar_i32_ptr)p)[i];   // address-space cast: C-style only
}

// Tiles of one row: KV heads x blocks of its visible context.
__device__ __forceinline__ int row_tiles(const DecodeArgs& a, int row) {
  int s, ctx;
  resolve_row(a, row, s, ctx);
  return ctx > 0 ? a.num_kv_heads * ((ctx + kBlockSize - 1) / kBlockSize) : 0;
}

// Prefix of tiles over rows in LDS: entry c is the first tile of row c * chunk
// (chunk = 1 up to kMaxRowsLds rows). Workgroup 0 also stores the per-row
// prefix in the workspace for the merge kernel. Returns the total tile count.
__device__ int build_tile_prefix(const DecodeArgs& a, int* s_pre, int* s_scan, int chunk, int nch) {
  const int tid = threadIdx.x;
  const int per = (nch + kThreads - 1) / kThreads;   // chunks per thread
  const int c0 = tid * per;
  int mine = 0;
  for (int c = c0; c < min(nch, c0 + per); ++c)
    for (int r = c * chunk; r < min(a.num_rows, (c + 1) * chunk); ++r) mine += row_tiles(a, r);
  s_scan[tid] = mine;
  __syncthreads();
  for (int off = 1; off < kThreads; off <<= 1) {
    const int v = tid >= off ? s_scan[tid - off] : 0;
    __syncthreads();
    s_scan[tid] += v;
    __syncthreads();
  }
  int run = s_scan[tid] - mine;
  for (int c = c0; c < min(nch, c0 + per); ++c) {
    s_pre[c] = run;
    for (int r = c * chunk; r < min(a.num_rows, (c + 1) * chunk); ++r) {
      if (blockIdx.x == 0) a.ws_rows[r] = run;
      run += row_tiles(a, r);
    }
  }
  if (tid == kThreads - 1) {
    s_pre[nch] = s_scan[kThreads - 1];
    if (blockIdx.x == 0) a.ws_rows[a.num_rows] = s_scan[kThreads - 1];
  }
  __syncthreads();
  return s_pre[nch];
}

// Where a worker stands: tile b of (row, KV head g). All fields are uniform.
struct Cursor {
  int row, s, ctx, nblk, dirv, g, b;
};

__device__ __forceinline__ void enter_row(const DecodeArgs& a, int row, Cursor& c) {
  c.row = row;
  resolve_row(a, row, c.s, c.ctx);
  c.nblk = c.ctx > 0 ? (c.ctx + kBlockSize - 1) / kBlockSize : 0;
  // Only the tail block has slots outside the context: its entry's direction.
  c.dirv = entry_direction(a.dir, a.cls, a.dir_per_entry, a.max_blocks_per_seq, c.s, c.nblk > 0 ? c.nblk - 1 : 0);
  c.row = __builtin_amdgcn_readfirstlane(c.row);
  c.s = __builtin_amdgcn_readfirstlane(c.s);
  c.ctx = __builtin_amdgcn_readfirstlane(c.ctx);
  c.nblk = __builtin_amdgcn_readfirstlane(c.nblk);
  c.dirv = __builtin_amdgcn_readfirstlane(c.dirv);
}

// Next tile in (row, KV head, block) order; rows without context have no tiles.
// Only called while tiles remain in the worker's range, so a row exists.
__device__ __forceinline__ void advance(const DecodeArgs& a, Cursor& c) {
  if (++c.b < c.nblk) return;
  c.b = 0;
  if (++c.g < a.num_kv_heads) return;
  c.g = 0;
  int row = c.row;
  do {
    ++row;
    enter_row(a, row, c);
  } while (c.nblk == 0 && row + 1 < a.num_rows);
}

// Tile t (< total): binary search over the chunk prefix, then rows of the chunk.
__device__ void locate(const DecodeArgs& a, const int* s_pre, int chunk, int nch, int t, Cursor& c) {
  int ch = upper_index(s_pre, nch + 1, t);
  ch = min(ch, nch - 1);
  int base = s_pre[ch];
  int row = ch * chunk;
  for (;;) {
    enter_row(a, row, c);
    const int n = c.nblk * a.num_kv_heads;
    if (t < base + n || row + 1 >= a.num_rows) break;
    base += n;
    ++row;
  }
  const int local = t - base;
  c.g = __builtin_amdgcn_readfirstlane(c.nblk > 0 ? local / c.nblk : 0);
  c.b = __builtin_amdgcn_readfirstlane(local - c.g * c.nblk);
}

__device__ __forceinline__ int worker_of(int64_t tile, int64_t total, int64_t workers) {
  return (int)(((tile + 1) * workers - 1) / total);
}

template <int G>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void decode_mfma_kernel(DecodeArgs a) {
  static_assert(G >= 1 && G <= 16, "heads of a group must fit the 16 MFMA columns");
  __shared__ int s_pre[kMaxRowsLds + 1];
  __shared__ int s_scan[kThreads];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int grp = lane >> 4;
  const int col = lane & 15;
  const bool head_lane = col < G;
  const int nkv = a.num_kv_heads;
  const int Hq = a.num_q_heads;

  const int chunk = (a.num_rows + kMaxRowsLds - 1) / kMaxRowsLds;
  const int nch = (a.num_rows + chunk - 1) / chunk;
  const int total = build_tile_prefix(a, s_pre, s_scan, chunk, nch);

  // This wave's share of the tiles; with fewer tiles than waves the last waves
  // idle, so every worker has at least one tile.
  const int workers = min(a.num_workers, total);
  const int wid = blockIdx.x * kWaves + wave_id_uniform();
  if (wid >= workers) return;
  const int t0 = (int)((int64_t)wid * total / workers);
  const int t1 = (int)((int64_t)(wid + 1) * total / workers);
  const int n = t1 - t0;

  const uint32_t k_lane = (uint32_t)col * kHeadDim + 8 * grp;        // + 32 c
  const uint32_t v_lane = (uint32_t)(4 * grp) * kHeadDim + 8 * col;  // + j * kHeadDim
  // kDepth K/V register sets: tile i uses set i % kDepth while the loads of
  // tiles i + 1 .. i + kDepth - 1 are in flight in the others, and tile
  // i + kDepth's are issued into set i % kDepth as soon as its registers are
  // read.
  v4u_t qf[4], kf_[kDepth][4], vf_[kDepth][4];
  floatx4_t acc[8];
  float m_ref = kNoMax, l_part = 0.0f;

  auto table = [&](const Cursor& c) -> int {
    const int blk = load_uniform(a.block_tables, (size_t)c.s * a.max_blocks_per_seq + c.b);
    return (blk >= 0 && blk < a.num_blocks) ? blk : -1;
  };
  // Slots of tile c that hold context: all 16, except in a tail block, where
  // they are [0, r) walking from the left and [16 - r, 16) from the right.
  // The rows of the other slots are not loaded (their scores and V rows are
  // dropped by selection in the tile's body whatever the registers hold).
  auto slot_lo = [&](const Cursor& c) -> int {
    const int r = c.ctx & (kBlockSize - 1);
    return (c.b == c.nblk - 1 && r != 0 && c.dirv < 0) ? kBlockSize - r : 0;
  };
  auto slot_hi = [&](const Cursor& c) -> int {
    const int r = c.ctx & (kBlockSize - 1);
    return (c.b == c.nblk - 1 && r != 0 && c.dirv > 0) ? r : kBlockSize;
  };
  auto issue_k = [&](v4u_t (&kf)[4], int blk, const Cursor& c) {
    if (blk < 0) return;
    if (col < slot_lo(c) || col >= slot_hi(c)) return;   // this lane's K row is slot col
    const size_t base = ((size_t)blk * nkv + c.g) * kTileElems + k_lane;
#pragma unroll
    for (int k = 0; k < 4; ++k) kf[k] = load_nt(a.k_pool, base + 32 * k);
  };
  auto issue_v = [&](v4u_t (&vf)[4], int blk, const Cursor& c) {
    if (blk < 0) return;
    const int lo = slot_lo(c), hi = slot_hi(c);
    const size_t base = ((size_t)blk * nkv + c.g) * kTileElems + v_lane;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int slot = 4 * grp + j;   // this lane's V rows
      if (slot >= lo && slot < hi) vf[j] = load_nt(a.v_pool, base + (size_t)j * kHeadDim);
    }
  };
  auto load_q = [&](const Cursor& c) {
    const size_t qoff = ((size_t)c.row * Hq + c.g * G + col) * kHeadDim + 8 * grp;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      qf[k] = v4u_t{0u, 0u, 0u, 0u};
      if (head_lane) qf[k] = *reinterpret_cast<const v4u_t*>(static_cast<const uint16_t*>(a.q) + qoff + 32 * k);
    }
  };

  // cur[d] / blk[d]: tile i + d (entries read one tile before their loads issue)
  Cursor cur[kDepth + 2];
  int blk[kDepth + 2];
  locate(a, s_pre, chunk, nch, t0, cur[0]);
  blk[0] = table(cur[0]);
  issue_k(kf_[0], blk[0], cur[0]);
  issue_v(vf_[0], blk[0], cur[0]);
  load_q(cur[0]);
  bool whole = cur[0].b == 0;   // this wave saw the segment's first tile
#pragma unroll
  for (int d = 1; d <= kDepth; ++d) {
    cur[d] = cur[d - 1];
    blk[d] = -1;
    if (d < n) {
      advance(a, cur[d]);
      blk[d] = table(cur[d]);
      if (d < kDepth) {
        issue_k(kf_[d], blk[d], cur[d]);
        issue_v(vf_[d], blk[d], cur[d]);
      }
    }
  }
  blk[kDepth + 1] = -1;
  cur[kDepth + 1] = cur[kDepth];
#pragma unroll
  for (int t = 0; t < 8; ++t) acc[t] = floatx4_t{0.0f, 0.0f, 0.0f, 0.0f};

  // Tile i, its K/V in (kf, vf).
  auto body = [&](int i, v4u_t (&kf)[4], v4u_t (&vf)[4]) __attribute__((always_inline)) {
    Cursor& c0 = cur[0];
    const int blk0 = blk[0];
    // the tile kDepth + 1 ahead: its table entry is read now, used one tile later
    cur[kDepth + 1] = cur[kDepth];
    blk[kDepth + 1] = -1;
    if (i + kDepth + 1 < n) {
      advance(a, cur[kDepth + 1]);
      blk[kDepth + 1] = table(cur[kDepth + 1]);
    }
    floatx4_t sc = {0.0f, 0.0f, 0.0f, 0.0f};
    if (blk0 >= 0) {
#pragma unroll
      for (int k = 0; k < 4; ++k)
        sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kf[k]),
                                                     __builtin_bit_cast(bf16x8_t, qf[k]), sc, 0, 0, 0);
    }
    const bool seg_end = c0.b == c0.nblk - 1 || i + 1 == n;
    if (i + 1 == n) {
      // this worker's entry of the cut list: the segment it started and
      // leaves unfinished (the merge folds it), else -1
      const bool starts_cut = whole && c0.b != c0.nblk - 1;
      if (lane == 0) a.ws_cut[wid] = starts_cut ? c0.row * nkv + c0.g : -1;
    }
    // K and query registers are free: keys kDepth tiles ahead (and the query
    // of the next tile's segment)
    if (i + kDepth < n) issue_k(kf, blk[kDepth], cur[kDepth]);
    if (i + 1 < n && seg_end) load_q(cur[1]);
    if (blk0 >= 0) {
      float s[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) s[r] = sc[r] * a.scale_log2;
      if (c0.b == c0.nblk - 1 && (c0.ctx & (kBlockSize - 1)) != 0) {   // tail: drop slots past the context
        const int gt = lane_id_here() >> 4;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          if (c0.b * kBlockSize + slot_of_offset(4 * gt + r, c0.dirv) >= c0.ctx) {
            s[r] = -INFINITY;
            vf[r] = v4u_t{0u, 0u, 0u, 0u};
          }
        }
      }
      float mx = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
      if (__builtin_amdgcn_ballot_w64(head_lane && mx > m_ref + kRescaleSlack) != 0) {
        // rare: move each head's reference max to the max over its 16 slots
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_ref, mx);
        const float alpha = fast_exp2(m_ref - m_new);
        m_ref = m_new;
        l_part *= alpha;
#pragma unroll
        for (int t = 0; t < 8; ++t) {
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[t][r] *= alpha;
        }
      }
      float p[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) p[r] = fast_exp2(s[r] - m_ref);
      l_part += (p[0] + p[1]) + (p[2] + p[3]);
      const short4_t pb = __builtin_bit_cast(short4_t, uint2{pack2_bf16(p[0], p[1]), pack2_bf16(p[2], p[3])});
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const uint32_t sel = (t & 1) ? 0x07060302u : 0x05040100u;
        const uint32_t lo = __builtin_amdgcn_perm(vf[1][t >> 1], vf[0][t >> 1], sel);
        const uint32_t hi = __builtin_amdgcn_perm(vf[3][t >> 1], vf[2][t >> 1], sel);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(short4_t, uint2{lo, hi}), pb, acc[t], 0, 0, 0);
      }
    }
    // V registers are free: values kDepth tiles ahead
    if (i + kDepth < n) issue_v(vf, blk[kDepth], cur[kDepth]);

    if (seg_end) {
      // The four lane groups of a head hold disjoint slots: total their weights.
      float l_head = l_part;
      l_head += __shfl_xor(l_head, 16);
      l_head += __shfl_xor(l_head, 32);
      const bool direct = whole && c0.b == c0.nblk - 1;   // the whole segment was this wave's
      if (head_lane) {
        const int h = c0.g * G + col;
        if (direct) {
          const float inv = l_head > 0.0f ? 1.0f / l_head : 0.0f;
          uint16_t* o = static_cast<uint16_t*>(a.out) + ((size_t)c0.row * Hq + h) * kHeadDim + 32 * grp;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const v4u_t w4 = v4u_t{pack2_bf16(acc[0][r] * inv, acc[1][r] * inv), pack2_bf16(acc[2][r] * inv, acc[3][r] * inv),
                                   pack2_bf16(acc[4][r] * inv, acc[5][r] * inv), pack2_bf16(acc[6][r] * inv, acc[7][r] * inv)};
            *reinterpret_cast<v4u_t*>(o + 8 * r) = w4;
          }
        } else {
          const size_t slot = ((size_t)c0.row * nkv + c0.g + wid) * G + col;   // partial (segment + worker)
          float* dst = a.ws_acc + slot * kHeadDim + 32 * grp;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            *reinterpret_cast<floatx4_t*>(dst + 8 * r) = floatx4_t{acc[0][r], acc[1][r], acc[2][r], acc[3][r]};
            *reinterpret_cast<floatx4_t*>(dst + 8 * r + 4) = floatx4_t{acc[4][r], acc[5][r], acc[6][r], acc[7][r]};
          }
          if (grp == 0) {
            a.ws_ml[2 * slot] = m_ref;
            a.ws_ml[2 * slot + 1] = l_head;
          }
        }
      }
      m_ref = kNoMax;
      l_part = 0.0f;
#pragma unroll
      for (int t = 0; t < 8; ++t) acc[t] = floatx4_t{0.0f, 0.0f, 0.0f, 0.0f};
      whole = true;
    }
#pragma unroll
    for (int d = 0; d <= kDepth; ++d) {
      cur[d] = cur[d + 1];
      blk[d] = blk[d + 1];
    }
  };
  auto group = [&](int i, auto dc) __attribute__((always_inline)) -> bool {
    constexpr int d = decltype(dc)::value;
    if (i + d >= n) return false;
    body(i + d, kf_[d], vf_[d]);
    return true;
  };
#pragma clang loop unroll(disable)
  for (int i = 0; i < n; i += kDepth) {
    if (!group(i, std::integral_constant<int, 0>{}) || !group(i, std::integral_constant<int, 1>{})) break;
    if constexpr (kDepth > 2) {
      if (!group(i, std::integral_constant<int, 2>{})) break;
    }
    if constexpr (kDepth > 3) {
      if (!group(i, std::integral_constant<int, 3>{})) break;
    }
  }
}

// Segments cut between workers: o = sum_w 2^(m_w - M) acc_w / sum_w 2^(m_w -
// M) l_w over the partials of workers w0 .. w1. The decode kernel's worker
// w0 (the one that started the segment and left it unfinished) named the
// segment in its entry of the cut list; every other entry is -1, so the merge
// grid has one wave per worker and most waves return after one load. Segments
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
  const int total = a.ws_rows[a.num_rows];
  const int workers = min(a.num_workers, total);
  if (item >= workers) return;
  const int code = a.ws_cut[item];
  if (code < 0) return;
  const int nkv = a.num_kv_heads;
  const int row = __builtin_amdgcn_readfirstlane(code / nkv);
  const int g = __builtin_amdgcn_readfirstlane(code - (code / nkv) * nkv);
  int s, ctx;
  resolve_row(a, row, s, ctx);
  const int nblk = (ctx + kBlockSize - 1) / kBlockSize;
  const int64_t first_tile = (int64_t)a.ws_rows[row] + (int64_t)g * nblk;
  const int w0 = item;
  const int w1 = __builtin_amdgcn_readfirstlane(worker_of(first_tile + nblk - 1, total, workers));
  const int hl = lane / L, sub = lane % L;
  const size_t seg = (size_t)row * nkv + g;
  // the head's max over the partials (lanes of the head take every L-th one)
  float M = kNoMax;
  for (int w = w0 + sub; w <= w1; w += L) M = fmaxf(M, a.ws_ml[2 * ((seg + w) * G + hl)]);
#pragma unroll
  for (int o = L / 2; o >= 1; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
  float Lsum = 0.0f;
  float acc[DPL];
#pragma unroll
  for (int d = 0; d < DPL; ++d) acc[d] = 0.0f;
  for (int c = w0; c <= w1; c += L) {
    // lane sub holds the weight of partial c + sub of its head
    float wt = 0.0f;
    if (c + sub <= w1) {
      const size_t slot = (seg + c + sub) * G + hl;
      wt = fast_exp2(a.ws_ml[2 * slot] - M);
      Lsum = fmaf(a.ws_ml[2 * slot + 1], wt, Lsum);
    }
    const int cnt = min(L, w1 - c + 1);
    for (int j0 = 0; j0 < cnt; j0 += 8) {
      float2 v[8][DPL / 2];
      float wj[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {   // indices clamped in range; padding gets weight 0
        const int j = min(j0 + u, cnt - 1);
        const float w = __shfl(wt, hl * L + j);
        wj[u] = (j0 + u < cnt) ? w : 0.0f;
        const float2* src = reinterpret_cast<const float2*>(a.ws_acc + ((seg + c + j) * G + hl) * kHeadDim + sub * DPL);
#pragma unroll
        for (int q = 0; q < DPL / 2; ++q) v[u][q] = src[q];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
#pragma unroll
        for (int q = 0; q < DPL / 2; ++q) {
          acc[2 * q] = fmaf(v[u][q].x, wj[u], acc[2 * q]);
          acc[2 * q + 1] = fmaf(v[u][q].y, wj[u], acc[2 * q + 1]);
        }
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

}  // namespace

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

template <int G>
hipError_t launch_group(DecodeArgs a, hipStream_t stream, int slot) {
  int grid = resident_workgroups(reinterpret_cast<const void*>(&decode_mfma_kernel<G>), kThreads, slot, stream);
  grid = grid < kMaxDecodeGrid ? grid : kMaxDecodeGrid;
  a.num_workers = grid * kWaves;
  hipLaunchKernelGGL((decode_mfma_kernel<G>), dim3(grid), dim3(kThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // one wave per worker (its cut-list entry) and per row (rows without context)
  const long long items = a.num_workers > a.num_rows ? a.num_workers : a.num_rows;
  const unsigned merge_grid = (unsigned)((items + kMergeWaves - 1) / kMergeWaves);
  hipLaunchKernelGGL(decode_mfma_merge_kernel<G>, dim3(merge_grid), dim3(kMergeWaves * kWave), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

DecodePlan plan_decode(int32_t num_rows, int32_t max_ctx) {
  DecodePlan p;
  const int64_t maxblk = max_ctx > 0 ? ((int64_t)max_ctx + kBlockSize - 1) / kBlockSize : 1;
  int sb = kMaxSplitBlocks;   // 1024 tokens per split by default
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
           round_up_256(slots * 2 * sizeof(float)) + (size_t)kWaves * kMaxDecodeGrid * sizeof(int32_t);
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
    return;
  }
  a.ws_rows = nullptr;
  a.ws_cut = nullptr;
  a.ws_acc = reinterpret_cast<float*>(base);
  a.ws_ml = base ? a.ws_acc + (size_t)a.num_rows * a.num_q_heads * a.n_split_max * kHeadDim : nullptr;
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
