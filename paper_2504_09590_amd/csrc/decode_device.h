// Device code of the bf16 decode on the matrix cores, shared by the decode
// launch (decode.hip) and the fused prefill|decode launch (mixed.hip).
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

#pragma once

#include "decode_common.h"

#include <type_traits>

namespace bros {
namespace dm {

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
// Each thread totals a run of consecutive chunks, parking each chunk's count
// in its own entry; a scan within each wave and one across the waves (one
// barrier) gives every thread its start, and the thread turns its entries
// into prefixes. `s_scan` holds kThreads / kWave ints.
static __device__ int build_tile_prefix(const DecodeArgs& a, int* s_pre, int* s_scan, int chunk, int nch) {
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1), w = tid / kWave;
  const int per = (nch + kThreads - 1) / kThreads;   // chunks per thread
  const int c0 = tid * per, c1 = min(nch, c0 + per);
  int mine = 0;
  for (int c = c0; c < c1; ++c) {
    int t = 0;
    for (int r = c * chunk; r < min(a.num_rows, (c + 1) * chunk); ++r) t += row_tiles(a, r);
    s_pre[c] = t;   // (this thread's entry: its count for now)
    mine += t;
  }
  int inc = mine;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int u = __shfl_up(inc, o);
    if (lane >= o) inc += u;
  }
  if (lane == kWave - 1) s_scan[w] = inc;
  __syncthreads();
  int run = inc - mine, total = 0;
#pragma unroll
  for (int i = 0; i < kThreads / kWave; ++i) {
    const int x = s_scan[i];
    run += i < w ? x : 0;
    total += x;
  }
  for (int c = c0; c < c1; ++c) {
    const int t = s_pre[c];
    s_pre[c] = run;
    if (blockIdx.x == 0) {
      if (chunk == 1) {
        a.ws_rows[c] = run;
      } else {
        int rr = run;
        for (int r = c * chunk; r < min(a.num_rows, (c + 1) * chunk); ++r) {
          a.ws_rows[r] = rr;
          rr += row_tiles(a, r);
        }
      }
    }
    run += t;
  }
  if (tid == kThreads - 1) {
    s_pre[nch] = total;
    if (blockIdx.x == 0) a.ws_rows[a.num_rows] = total;
  }
  __syncthreads();
  return total;
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
static __device__ void locate(const DecodeArgs& a, const int* s_pre, int chunk, int nch, int t, Cursor& c) {
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


// One worker's share: tiles [t0, t0 + n) of the (row, KV head, block) order
// (n >= 1), the tile prefix over rows in LDS (s_pre, chunk, nch) as
// build_tile_prefix left it. Run by one wave; `wid` names its partial slots.
// With `workers` > 0 the shares are the even split of `total` tiles over
// `workers` workers, so the worker holding any tile is known in closed form;
// 0 leaves that to the merge.
template <int G>
__device__ __forceinline__ void decode_worker(const DecodeArgs& a, const int* s_pre, int chunk, int nch, int wid,
                                              int t0, int n, int total, int workers) {
  static_assert(G >= 1 && G <= 16, "heads of a group must fit the 16 MFMA columns");
  const int lane = threadIdx.x & (kWave - 1);
  const int grp = lane >> 4;
  const int col = lane & 15;
  const bool head_lane = col < G;
  const int nkv = a.num_kv_heads;
  const int Hq = a.num_q_heads;

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
      // leaves unfinished (the merge folds it), else -1; and the worker that
      // holds the segment's last tile, the largest w with
      // floor(w total / workers) <= that tile (-1: the merge finds it)
      const bool starts_cut = whole && c0.b != c0.nblk - 1;
      int w1 = -1;
      if (starts_cut && workers > 0) {
        const int64_t last = (int64_t)t0 + i + (c0.nblk - 1 - c0.b);
        w1 = (int)(((last + 1) * workers - 1) / total);
      }
      if (lane == 0) {
        a.ws_cut[2 * wid] = starts_cut ? c0.row * nkv + c0.g : -1;
        a.ws_cut[2 * wid + 1] = w1;
      }
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

}  // namespace dm
}  // namespace bros
