// fp32 decode on the vector ALU: split-K paged attention over the
// bidirectional pool (the bf16 path runs on the matrix cores, decode.hip).
//
// What it computes (Sec. 2.1 decode attention over the cached KV; Sec. 5.1
// bidirectional slot order; Sec. 6 direction-aware paged kernel): for query
// row r of sequence s and query head h in KV group g = h / G,
//     out[r][h] = sum_p softmax_p(scale * q[r][h] . K[p][g]) V[p][g],  p < ctx(r).
// fp32 products and sums throughout (the fp32 tolerance is 1e-5).
//
// Work. An item is (row, KV head, split of up to `split_blocks` blocks). A
// persistent grid walks the item list, workgroup w taking items w, w + grid,
// ...; each workgroup first builds, in LDS, the prefix count of items per
// row, so an item index maps to its row by binary search.
//
// Inside an item, a "stream" (one wave, or for G = 8 a pair of waves each
// taking four of the eight heads) walks every NSTREAM-th block of the split.
// A (block, KV head) tile is 16 slots x 128 head dims, contiguous in the pool
// ([num_blocks][Hkv][16][128]); lane (R = lane / 16, C = lane % 16) holds
// slots R, R+4, R+8, R+12 and head dims [8C, 8C+8). The next block's K is
// requested as soon as this block's scores are formed, its V as soon as this
// block's PV product is done, across item boundaries.
//
// Per block, within each 16-lane row (one DPP row):
//   1. QK partials over the lane's 8 dims for its 4 slots x GW heads;
//   2. a transposing butterfly (mirror, half-mirror, quad swaps): at every
//      stage a lane keeps half of its values and adds its partner's copy of
//      them, so after four stages lane C holds complete scores of its own
//      (head, slot) pairs instead of all 4GW scores replicated;
//   3. online softmax in base 2 on those few scores. The running reference
//      max of a (row, head) is only moved when a score exceeds it by more than
//      2^8, so the rescale of the accumulators is rare; weights stay <= 256;
//   4. the weights are broadcast back across the row (row_newbcast) and PV
//      accumulates with fused multiply-adds.
// Direction only decides which physical slots hold valid positions (see
// decode.hip). Rows of a wave, then streams of the workgroup (through LDS),
// then splits (merge kernel) are combined with max-rescaling.
#include "decode_common.h"

namespace bros {
namespace {

constexpr int kSlotF32Base = 4;   // resident_workgroups cache slots 4..7

constexpr int ilog2(int x) { return x <= 1 ? 0 : 1 + ilog2(x / 2); }

// DPP row controls of the four butterfly stages; stage k pairs lanes that
// differ in bit 3 - k of C (and possibly lower bits), see stage_side().
constexpr int kStageCtrl[4] = {0x140, 0x141, 0x4e, 0xb1};  // row_mirror, row_half_mirror, quad ^2, quad ^1
__device__ __forceinline__ int stage_side(int C, int k) { return (C >> (3 - k)) & 1; }

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __builtin_amdgcn_update_dpp(0.0f, x, CTRL, 0xf, 0xf, false);
}
template <int LANE>
__device__ __forceinline__ float row_bcast(float x) {   // lane LANE of each row -> whole row
  return __builtin_amdgcn_update_dpp(0.0f, x, 0x150 + LANE, 0xf, 0xf, false);
}
__device__ __forceinline__ float row_bcast_dyn(float x, int lane) {   // lane is a compile-time constant after unrolling
  switch (lane) {
    case 0: return row_bcast<0>(x);
    case 1: return row_bcast<1>(x);
    case 2: return row_bcast<2>(x);
    case 3: return row_bcast<3>(x);
    case 4: return row_bcast<4>(x);
    case 5: return row_bcast<5>(x);
    case 6: return row_bcast<6>(x);
    case 7: return row_bcast<7>(x);
    case 8: return row_bcast<8>(x);
    case 9: return row_bcast<9>(x);
    case 10: return row_bcast<10>(x);
    case 11: return row_bcast<11>(x);
    case 12: return row_bcast<12>(x);
    case 13: return row_bcast<13>(x);
    case 14: return row_bcast<14>(x);
    default: return row_bcast<15>(x);
  }
}

// Eight consecutive head dims of one slot (or of one query row).
struct Frag {
  float f[8];
  __device__ void load(const void* base, size_t elem) {
    const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(base) + elem);
    const float4 a = p[0], b = p[1];
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w; f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
  }
  __device__ void zero() {
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = 0.0f;
  }
  __device__ float dot(const Frag& k) const {
    float acc = f[0] * k.f[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) acc = fmaf(f[i], k.f[i], acc);
    return acc;
  }
};

__device__ __forceinline__ int splits_of(int ctx, int sb) {
  return ctx <= 0 ? 1 : ((ctx + kBlockSize - 1) / kBlockSize + sb - 1) / sb;
}

// The scores of one (row of 16 lanes, block): v = 4 * head + j for slot R + 4j.
template <int GW>
struct Layout {
  static constexpr int NV = 4 * GW;                         // scores per lane row
  static constexpr int NPL = NV >= 16 ? NV / 16 : 1;        // scores a lane ends up holding
  static constexpr int NHALVE = ilog2(NV) < 4 ? ilog2(NV) : 4;
  static constexpr int DUP = NV >= 16 ? 1 : 16 / NV;        // lanes holding the same score
  static constexpr int GROUP = 16 / GW;                     // lanes holding one head's scores
};

// Online softmax state of one wave for GW query heads over one item.
template <int GW>
struct WaveState {
  using LY = Layout<GW>;
  float m_ref;        // reference max of this lane's head (log2 units)
  float l_part;       // sum of this lane's own weights (primary lanes only)
  float acc[GW][8];   // unnormalised outputs, head dims [8C, 8C+8), this lane row's slots

  __device__ void reset() {
    m_ref = kNoMax;
    l_part = 0.0f;
#pragma unroll
    for (int h = 0; h < GW; ++h) {
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] = 0.0f;
    }
  }

  // Scores of this lane's (head, slot) pairs, already in log2 units.
  __device__ void scores(const Frag (&q)[GW], const Frag (&kf)[4], float scale_log2, int C,
                         float (&sc)[LY::NPL]) const {
    constexpr int NV = LY::NV, NHALVE = LY::NHALVE;
    float part[NV];
#pragma unroll
    for (int h = 0; h < GW; ++h) {
#pragma unroll
      for (int j = 0; j < 4; ++j) part[4 * h + j] = q[h].dot(kf[j]);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int n = NV >> k;
      if (k < NHALVE) {
        const bool side = stage_side(C, k);
#pragma unroll
        for (int i = 0; i < n / 2; ++i) {
          const float keep = side ? part[i + n / 2] : part[i];
          const float send = side ? part[i] : part[i + n / 2];
          float recv;
          if (k == 0) recv = dpp<kStageCtrl[0]>(send);
          else if (k == 1) recv = dpp<kStageCtrl[1]>(send);
          else if (k == 2) recv = dpp<kStageCtrl[2]>(send);
          else recv = dpp<kStageCtrl[3]>(send);
          part[i] = keep + recv;
        }
      } else {   // fewer scores than lanes: plain all-reduce on the one left
        part[0] += (k == 2) ? dpp<kStageCtrl[2]>(part[0]) : dpp<kStageCtrl[3]>(part[0]);
      }
    }
#pragma unroll
    for (int i = 0; i < LY::NPL; ++i) sc[i] = part[i] * scale_log2;
  }

  // Softmax update with this block's scores, then PV with its V fragments.
  __device__ void update(float (&sc)[LY::NPL], const Frag (&vf)[4], bool primary) {
    constexpr int NPL = LY::NPL, DUP = LY::DUP, GROUP = LY::GROUP;
    float mx = sc[0];
#pragma unroll
    for (int i = 1; i < NPL; ++i) mx = fmaxf(mx, sc[i]);
    if (GROUP >= 2) mx = fmaxf(mx, dpp<0xb1>(mx));
    if (GROUP >= 4) mx = fmaxf(mx, dpp<0x4e>(mx));
    if (GROUP >= 8) mx = fmaxf(mx, dpp<0x141>(mx));
    if (GROUP >= 16) mx = fmaxf(mx, dpp<0x140>(mx));
    if (__builtin_amdgcn_ballot_w64(mx > m_ref + kRescaleSlack) != 0) {
      const float m_new = fmaxf(m_ref, mx);
      const float alpha = fast_exp2(m_ref - m_new);
      l_part *= alpha;
      m_ref = m_new;
#pragma unroll
      for (int h = 0; h < GW; ++h) {
        const float ah = GW == 1 ? alpha : row_bcast_dyn(alpha, h * GROUP);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] *= ah;
      }
    }
    float p[NPL];
    float psum = 0.0f;
#pragma unroll
    for (int i = 0; i < NPL; ++i) {
      p[i] = fast_exp2(sc[i] - m_ref);
      psum += p[i];
    }
    l_part += primary ? psum : 0.0f;
    // Weight v = 4h + j lives on lane (v / NPL) * DUP of the row.
#pragma unroll
    for (int h = 0; h < GW; ++h) {
      float wv[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) wv[j] = row_bcast_dyn(p[(4 * h + j) % NPL], ((4 * h + j) / NPL) * DUP);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float t = fmaf(wv[0], vf[0].f[e], acc[h][e]);
        t = fmaf(wv[1], vf[1].f[e], t);
        t = fmaf(wv[2], vf[2].f[e], t);
        acc[h][e] = fmaf(wv[3], vf[3].f[e], t);
      }
    }
  }

  // Per-head (m, l) to every lane, then the four rows of the wave merged:
  // afterwards every row holds the wave's totals for its head dims.
  __device__ void merge_rows(float (&mh)[GW], float (&lh)[GW]) {
    constexpr int GROUP = LY::GROUP;
    float l_head = l_part;
    if (GROUP >= 2) l_head += dpp<0xb1>(l_head);
    if (GROUP >= 4) l_head += dpp<0x4e>(l_head);
    if (GROUP >= 8) l_head += dpp<0x141>(l_head);
    if (GROUP >= 16) l_head += dpp<0x140>(l_head);
#pragma unroll
    for (int h = 0; h < GW; ++h) {
      mh[h] = row_bcast_dyn(m_ref, h * GROUP);
      lh[h] = row_bcast_dyn(l_head, h * GROUP);
    }
#pragma unroll
    for (int xo = 16; xo <= 32; xo <<= 1) {
#pragma unroll
      for (int h = 0; h < GW; ++h) {
        const float mo = __shfl_xor(mh[h], xo);
        const float lo = __shfl_xor(lh[h], xo);
        const float M = fmaxf(mh[h], mo);
        const float a1 = fast_exp2(mh[h] - M), a2 = fast_exp2(mo - M);
        lh[h] = lh[h] * a1 + lo * a2;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = acc[h][e] * a1 + __shfl_xor(acc[h][e], xo) * a2;
        mh[h] = M;
      }
    }
  }
};

// One item as a stream sees it.
struct Item {
  int row, s, g, split, ctx, nblk, nsp, b_begin, nbw, dirv;
  int tbl;   // per lane: table entry of block b_begin + lane (or -1)
};

// Items per row (KV heads x splits) and their prefix, row-major and within a
// row KV-head-major, in LDS when the rows fit. Returns the number of items, or
// the size of a padded item space (empty items skipped) when they do not.
__device__ int build_item_prefix(const DecodeArgs& a, int* s_prefix, int* s_scan) {
  const int tid = threadIdx.x;
  const int nkv = a.num_kv_heads;
  if (a.num_rows > kMaxRowsLds) return a.num_rows * nkv * a.n_split_max;
  const int per = (a.num_rows + kThreads - 1) / kThreads;
  const int r0 = tid * per;
  int mine = 0;
  for (int r = r0; r < min(a.num_rows, r0 + per); ++r) {
    int s, ctx;
    resolve_row(a, r, s, ctx);
    mine += nkv * splits_of(ctx, a.split_blocks);
  }
  s_scan[tid] = mine;
  __syncthreads();
  for (int off = 1; off < kThreads; off <<= 1) {   // inclusive scan of the per-thread sums
    const int v = tid >= off ? s_scan[tid - off] : 0;
    __syncthreads();
    s_scan[tid] += v;
    __syncthreads();
  }
  int run = s_scan[tid] - mine;
  for (int r = r0; r < min(a.num_rows, r0 + per); ++r) {
    s_prefix[r] = run;
    int s, ctx;
    resolve_row(a, r, s, ctx);
    run += nkv * splits_of(ctx, a.split_blocks);
  }
  if (tid == kThreads - 1) s_prefix[a.num_rows] = s_scan[kThreads - 1];
  __syncthreads();
  return s_prefix[a.num_rows];
}

// Item k as stream `stream` of NSTREAM sees it: its blocks are b_begin + stream,
// b_begin + stream + NSTREAM, ... (nbw of them); lane i holds the table entry of
// block b_begin + i.
template <int NSTREAM>
__device__ __forceinline__ void fetch_item(const DecodeArgs& a, const int* s_prefix, int k, int stream,
                                           int lane, Item& it) {
  const int nkv = a.num_kv_heads;
  const int SB = a.split_blocks;
  const bool use_prefix = a.num_rows <= kMaxRowsLds;
  int row, local;
  if (use_prefix) {
    row = upper_index(s_prefix, a.num_rows + 1, k);
    local = k - s_prefix[row];
  } else {
    row = k / (nkv * a.n_split_max);
    local = k - row * nkv * a.n_split_max;
  }
  it.row = row;
  resolve_row(a, row, it.s, it.ctx);
  it.nsp = splits_of(it.ctx, SB);
  const int per_g = use_prefix ? it.nsp : a.n_split_max;
  it.g = local / per_g;
  it.split = local - it.g * per_g;
  it.nblk = it.ctx > 0 ? (it.ctx + kBlockSize - 1) / kBlockSize : 0;
  it.b_begin = it.split * SB;
  const int nb = it.split < it.nsp ? max(0, min(it.nblk, it.b_begin + SB) - it.b_begin) : 0;
  it.nbw = nb > stream ? (nb - stream + NSTREAM - 1) / NSTREAM : 0;
  // Only the tail block has slots outside the context: its entry's direction.
  it.dirv = entry_direction(a.dir, a.cls, a.dir_per_entry, a.max_blocks_per_seq, it.s, it.nblk > 0 ? it.nblk - 1 : 0);
  // Every field but the table entry is the same on all lanes: keep them in
  // scalar registers so the vector registers go to KV fragments.
  it.row = __builtin_amdgcn_readfirstlane(it.row);
  it.s = __builtin_amdgcn_readfirstlane(it.s);
  it.g = __builtin_amdgcn_readfirstlane(it.g);
  it.split = __builtin_amdgcn_readfirstlane(it.split);
  it.ctx = __builtin_amdgcn_readfirstlane(it.ctx);
  it.nblk = __builtin_amdgcn_readfirstlane(it.nblk);
  it.nsp = __builtin_amdgcn_readfirstlane(it.nsp);
  it.b_begin = __builtin_amdgcn_readfirstlane(it.b_begin);
  it.nbw = __builtin_amdgcn_readfirstlane(it.nbw);
  it.dirv = __builtin_amdgcn_readfirstlane(it.dirv);
  it.tbl = -1;
  if (lane < nb) it.tbl = a.block_tables[(size_t)it.s * a.max_blocks_per_seq + it.b_begin + lane];
}

template <int G>
__global__ __launch_bounds__(kThreads) void decode_f32_kernel(DecodeArgs a) {
  constexpr int GW = G > 4 ? 4 : G;     // heads per wave
  constexpr int HS = G / GW;            // waves sharing a block stream
  constexpr int NSTREAM = kWaves / HS;  // block streams per workgroup
  using LY = Layout<GW>;

  __shared__ int s_prefix[kMaxRowsLds + 1];
  __shared__ float s_acc[kWaves][GW][kHeadDim];
  __shared__ float s_m[kWaves][GW], s_l[kWaves][GW];
  __shared__ int s_scan[kThreads];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int w = wave_id_uniform();
  const int R = lane >> 4;
  const int C = lane & 15;
  const int stream = w / HS;
  const int hh = w % HS;                 // which four heads of the group this wave owns
  const int nkv = a.num_kv_heads;
  const int Hq = a.num_q_heads;

  const int total = build_item_prefix(a, s_prefix, s_scan);
  auto fetch = [&](int k, Item& it) { fetch_item<NSTREAM>(a, s_prefix, k, stream, lane, it); };

  Frag q[GW];
  Frag kf[4], vf[4];
  WaveState<GW> st;
  const bool primary = (C & (LY::DUP - 1)) == 0;
  const size_t lane_off = (size_t)R * kHeadDim + 8 * C;

  auto issue_k = [&](const Item& it, int i) -> int {
    const int blk = read_lane_i32(it.tbl, stream + NSTREAM * i);
    if (blk < 0 || blk >= a.num_blocks) return -1;
    const size_t base = ((size_t)blk * nkv + it.g) * kTileElems + lane_off;
#pragma unroll
    for (int j = 0; j < 4; ++j) kf[j].load(a.k_pool, base + (size_t)(4 * j) * kHeadDim);
    return blk;
  };
  auto issue_v = [&](const Item& it, int i) {
    const int blk = read_lane_i32(it.tbl, stream + NSTREAM * i);
    if (blk < 0 || blk >= a.num_blocks) return;
    const size_t base = ((size_t)blk * nkv + it.g) * kTileElems + lane_off;
#pragma unroll
    for (int j = 0; j < 4; ++j) vf[j].load(a.v_pool, base + (size_t)(4 * j) * kHeadDim);
  };

  int k = blockIdx.x;
  Item cur, nxt;
  bool cur_ok = false;
  while (k < total) {   // find the first non-empty item (only the padded space has empties)
    fetch(k, cur);
    if (cur.split < cur.nsp) { cur_ok = true; break; }
    k += gridDim.x;
  }
  int blk_next = -1;   // table entry of the block whose K/V are in flight
  if (cur_ok && cur.nbw > 0) {
    blk_next = issue_k(cur, 0);
    issue_v(cur, 0);
  }

  while (cur_ok) {
    // next item of this workgroup
    int kn = k + gridDim.x;
    bool nxt_ok = false;
    while (kn < total) {
      fetch(kn, nxt);
      if (nxt.split < nxt.nsp) { nxt_ok = true; break; }
      kn += gridDim.x;
    }
    const int h0 = cur.g * G + hh * GW;   // first query head of this wave
#pragma unroll
    for (int h = 0; h < GW; ++h) q[h].load(a.q, ((size_t)cur.row * Hq + h0 + h) * kHeadDim + 8 * C);
    st.reset();

    for (int i = 0; i < cur.nbw; ++i) {
      const int blk = blk_next;
      const int b = cur.b_begin + stream + NSTREAM * i;   // logical block index
      const bool more_here = i + 1 < cur.nbw;
      const bool more_next = !more_here && nxt_ok && nxt.nbw > 0;
      float sc[LY::NPL];
      if (blk >= 0) st.scores(q, kf, a.scale_log2, C, sc);
      // K registers are free: request the next block's keys
      if (more_here) blk_next = issue_k(cur, i + 1);
      else if (more_next) blk_next = issue_k(nxt, 0);
      else blk_next = -1;
      if (blk >= 0) {
        if (b == cur.nblk - 1 && (cur.ctx & (kBlockSize - 1)) != 0) {   // tail: drop slots past the context
          const int lt = lane_id_here();
          const int Rt = lt >> 4, Ct = lt & 15;
          int vbase = 0;   // index v = 4 * head + j of this lane's first score
#pragma unroll
          for (int k = 0; k < LY::NHALVE; ++k) vbase += stage_side(Ct, k) * (LY::NV >> (k + 1));
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            if (b * kBlockSize + slot_of_offset(Rt + 4 * j, cur.dirv) >= cur.ctx) vf[j].zero();
          }
#pragma unroll
          for (int i2 = 0; i2 < LY::NPL; ++i2) {
            const int j = (vbase + i2) & 3;
            if (b * kBlockSize + slot_of_offset(Rt + 4 * j, cur.dirv) >= cur.ctx) sc[i2] = -INFINITY;
          }
        }
        st.update(sc, vf, primary);
      }
      // V registers are free: request the next block's values
      if (more_here) issue_v(cur, i + 1);
      else if (more_next) issue_v(nxt, 0);
    }

    // Combine the streams of the workgroup and write this item's result.
    float mh[GW], lh[GW];
    st.merge_rows(mh, lh);
    if (lane < 16) {
#pragma unroll
      for (int h = 0; h < GW; ++h) {
#pragma unroll
        for (int e = 0; e < 8; ++e) s_acc[w][h][8 * C + e] = st.acc[h][e];
      }
    }
    if (lane == 0) {
#pragma unroll
      for (int h = 0; h < GW; ++h) {
        s_m[w][h] = mh[h];
        s_l[w][h] = lh[h];
      }
    }
    __syncthreads();
    const int hbase = cur.g * G;
    for (int idx = tid; idx < G * kHeadDim; idx += kThreads) {
      const int h = idx / kHeadDim;           // head within the group
      const int d = idx - h * kHeadDim;
      const int hq4 = h / GW, hl = h - hq4 * GW;
      float M = kNoMax;
#pragma unroll
      for (int sidx = 0; sidx < NSTREAM; ++sidx) M = fmaxf(M, s_m[sidx * HS + hq4][hl]);
      float L = 0.0f, A = 0.0f;
#pragma unroll
      for (int sidx = 0; sidx < NSTREAM; ++sidx) {
        const int ww = sidx * HS + hq4;
        const float wt = fast_exp2(s_m[ww][hl] - M);
        L = fmaf(s_l[ww][hl], wt, L);
        A = fmaf(s_acc[ww][hl][d], wt, A);
      }
      const size_t qh = (size_t)cur.row * Hq + hbase + h;
      if (cur.nsp == 1) {
        static_cast<float*>(a.out)[qh * kHeadDim + d] = L > 0.0f ? A / L : 0.0f;
      } else {
        const size_t slot = qh * a.n_split_max + cur.split;
        a.ws_acc[slot * kHeadDim + d] = A;
        if (d == 0) {
          a.ws_ml[2 * slot] = M;
          a.ws_ml[2 * slot + 1] = L;
        }
      }
    }
    __syncthreads();

    if (!nxt_ok) break;
    if (cur.nbw == 0 && nxt.nbw > 0) {   // nothing was in flight for the next item yet
      blk_next = issue_k(nxt, 0);
      issue_v(nxt, 0);
    }
    cur = nxt;
    k = kn;
  }
}

// Combine the split partials of every (row, head) whose context needed more
// than one split: o = sum_i 2^(m_i - M) acc_i / sum_i 2^(m_i - M) l_i.
__global__ __launch_bounds__(kHeadDim) void decode_f32_merge_kernel(DecodeArgs a) {
  const int hq = blockIdx.x % a.num_q_heads;
  const int row = blockIdx.x / a.num_q_heads;
  const int d = threadIdx.x;
  int s, ctx;
  resolve_row(a, row, s, ctx);
  if (ctx <= 0) return;
  const int nblk = (ctx + kBlockSize - 1) / kBlockSize;
  const int nsp = (nblk + a.split_blocks - 1) / a.split_blocks;
  if (nsp <= 1) return;
  const size_t base = ((size_t)row * a.num_q_heads + hq) * a.n_split_max;
  float M = kNoMax;
  for (int i = 0; i < nsp; ++i) M = fmaxf(M, a.ws_ml[2 * (base + i)]);
  float L = 0.0f, A = 0.0f;
  for (int i = 0; i < nsp; ++i) {
    const float wt = fast_exp2(a.ws_ml[2 * (base + i)] - M);
    L = fmaf(a.ws_ml[2 * (base + i) + 1], wt, L);
    A = fmaf(a.ws_acc[(base + i) * kHeadDim + d], wt, A);
  }
  static_cast<float*>(a.out)[((size_t)row * a.num_q_heads + hq) * kHeadDim + d] = L > 0.0f ? A / L : 0.0f;
}

template <int G>
hipError_t launch_group_f32(const DecodeArgs& a, hipStream_t stream, int slot) {
  const long long padded = (long long)a.num_rows * a.num_kv_heads * a.n_split_max;
  const int resident = resident_workgroups(reinterpret_cast<const void*>(&decode_f32_kernel<G>), kThreads, slot, stream);
  const int grid = (int)(padded < resident ? padded : resident);
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL((decode_f32_kernel<G>), dim3(grid), dim3(kThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.n_split_max <= 1) return e;
  hipLaunchKernelGGL(decode_f32_merge_kernel, dim3((unsigned)(a.num_rows * a.num_q_heads)), dim3(kHeadDim), 0,
                     stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_decode_f32(const DecodeArgs& a, int group, hipStream_t stream) {
  switch (group) {
    case 1: return launch_group_f32<1>(a, stream, kSlotF32Base + 0);
    case 2: return launch_group_f32<2>(a, stream, kSlotF32Base + 1);
    case 4: return launch_group_f32<4>(a, stream, kSlotF32Base + 2);
    case 8: return launch_group_f32<8>(a, stream, kSlotF32Base + 3);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace bros
