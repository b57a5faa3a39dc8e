// bros_attn_decode on gfx950: split-K paged attention over the bidirectional pool.
//
// What it computes (Sec. 2.1 decode attention over the cached KV; Sec. 5.1
// bidirectional slot order; Sec. 6 direction-aware paged kernel): for query
// row r of sequence s and query head h in KV group g = h / G,
//     out[r][h] = sum_p softmax_p(scale * q[r][h] . K[p][g]) V[p][g],  p < ctx(r).
//
// Work. An item is (row, KV head, split of up to `split_blocks` blocks).
// The kernel is persistent: a grid sized to what the chip holds at four waves
// per SIMD walks the item list, workgroup w taking items w, w + grid, ... Each
// workgroup first builds, in LDS, the prefix count of items per row, so an
// item index maps to its row by binary search. Bandwidth on this chip tracks
// the number of resident waves, so the kernel keeps under 128 VGPRs.
//
// Inside an item, a "stream" (one wave, or for G = 8 a pair of waves each
// taking four of the eight heads) walks every NSTREAM-th block of the split.
// A (block, KV head) tile is 16 slots x 128 head dims, contiguous in the pool
// ([num_blocks][Hkv][16][128]), so each load instruction reads 1 KiB
// contiguous; lane (R = lane / 16, C = lane % 16) holds slots R, R+4, R+8,
// R+12 and head dims [8C, 8C+8). One K and one V register set are recycled:
// the next block's K is requested as soon as this block's scores are formed,
// its V as soon as this block's PV product is done; the next block may belong
// to the workgroup's next item, so the memory pipeline does not drain between
// items. KV tiles are read with non-temporal loads when one wave uses them;
// when two waves share a tile (G = 8) the loads stay cacheable.
//
// Per block, within each 16-lane row (one DPP row):
//   1. QK partials over the lane's 8 dims for its 4 slots x GW heads (dot2 on
//      bf16 pairs: products exact, one rounding per pair, fp32 accumulation);
//   2. a transposing butterfly (mirror, half-mirror, quad swaps): at every
//      stage a lane keeps half of its values and adds its partner's copy of
//      them, so after four stages lane C holds complete scores of its own
//      (head, slot) pairs instead of all 4GW scores replicated;
//   3. online softmax in base 2 on those few scores. The running reference
//      max of a (row, head) is only moved when a score exceeds it by more than
//      2^8, so the rescale of the accumulators is rare; weights stay <= 256;
//   4. the weights are broadcast back across the row (row_newbcast) and PV
//      runs as dot2 over slot pairs (V repacked with v_perm, weights rounded
//      to bf16), fp32 accumulation.
// Direction only decides which physical slots hold valid positions: attention
// is a sum over the cached tokens, so each score is paired with the V row of
// the same physical slot, and the logical position b*16 + (dir > 0 ? slot :
// 15 - slot) is compared with the context length in the tail block. Invalid
// slots are removed by selection (scores -inf, V zeroed), never by
// multiplication, so a peer request's tokens or NaNs there cannot leak.
// Rows of a wave, then streams of the workgroup (through LDS), then splits
// (merge kernel) are combined with max-rescaling.
#include "bros_device.h"
#include "bros_kernels.h"

#include <math.h>

#include <mutex>

namespace bros {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kTileElems = kBlockSize * kHeadDim;   // one (block, KV head) tile
constexpr float kRescaleSlack = 8.0f;               // log2 units: weights stay <= 2^8
constexpr float kNoMax = -1.0e30f;                  // finite "no score yet" reference
constexpr int kMaxRowsLds = 4096;                   // rows whose item prefix fits in LDS
constexpr int kMaxSplitBlocks = 64;                 // one table entry per lane

typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2_t;
typedef __attribute__((__vector_size__(2 * sizeof(float)))) float float2_t;
typedef unsigned v4u_t __attribute__((ext_vector_type(4)));

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

// Eight consecutive head-dim elements of one slot (or of one query row).
template <bool BF16> struct Frag;
template <> struct Frag<true> {
  uint32_t w[4];
  __device__ void load(const void* base, size_t elem) {
    const uint4 v = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + elem);
    w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
  }
  __device__ void load_stream(const void* base, size_t elem) {
    const v4u_t v = __builtin_nontemporal_load(reinterpret_cast<const v4u_t*>(static_cast<const uint16_t*>(base) + elem));
    w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
  }
  __device__ void zero() { w[0] = w[1] = w[2] = w[3] = 0u; }
  __device__ float dot(const Frag& k) const {
    // First pair in the three-operand form with an inline zero addend: the
    // builtin with a 0 addend becomes the tied-accumulator form plus a move.
    float acc;
    asm("v_dot2_f32_bf16 %0, %1, %2, 0" : "=v"(acc) : "v"(w[0]), "v"(k.w[0]));
#pragma unroll
    for (int i = 1; i < 4; ++i)
      acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w[i]), __builtin_bit_cast(bf16x2_t, k.w[i]), acc, false);
    return acc;
  }
};
template <> struct Frag<false> {
  float f[8];
  __device__ void load(const void* base, size_t elem) {
    const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(base) + elem);
    const float4 a = p[0], b = p[1];
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w; f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
  }
  __device__ void load_stream(const void* base, size_t elem) { load(base, elem); }
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

template <bool BF16>
__device__ __forceinline__ void store_out(void* out, size_t elem, float v) {
  if constexpr (BF16) static_cast<uint16_t*>(out)[elem] = (uint16_t)f32_to_bf16_bits(v);
  else static_cast<float*>(out)[elem] = v;
}

// Lane id through an asm the compiler cannot hoist: values derived from it are
// recomputed where they are used instead of being held in registers.
__device__ __forceinline__ int lane_id_here() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {   // round to nearest even
  const float2_t f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

// Query row -> (sequence, visible context). Decode mode: row r is sequence r.
// Row mode: row r is a prefill row and sees its causal prefix.
__device__ __forceinline__ void resolve_row(const DecodeArgs& a, int row, int& s, int& ctx) {
  if (a.cu_q == nullptr) {
    s = row;
    ctx = a.ctx_lens[s];
  } else {
    s = min(upper_index(a.cu_q, a.num_seqs + 1, row), a.num_seqs - 1);
    ctx = a.ctx_lens[s] - (a.cu_q[s + 1] - row) + 1;
  }
  ctx = min(ctx, a.max_ctx);
  ctx = min(ctx, a.max_blocks_per_seq * kBlockSize);
}

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
template <int GW, bool BF16>
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
  __device__ void scores(const Frag<BF16> (&q)[GW], const Frag<BF16> (&kf)[4], float scale_log2, int C,
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
  __device__ void update(float (&sc)[LY::NPL], const Frag<BF16> (&vf)[4], bool primary) {
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
    // Weight v = 4h + j lives on lane (v / NPL) * DUP of the row; fetch each
    // head's four and (bf16) pack them in slot pairs right away.
    if constexpr (BF16) {
      uint32_t p01[GW], p23[GW];
#pragma unroll
      for (int h = 0; h < GW; ++h) {
        const float w0 = row_bcast_dyn(p[(4 * h + 0) % NPL], ((4 * h + 0) / NPL) * DUP);
        const float w1 = row_bcast_dyn(p[(4 * h + 1) % NPL], ((4 * h + 1) / NPL) * DUP);
        const float w2 = row_bcast_dyn(p[(4 * h + 2) % NPL], ((4 * h + 2) / NPL) * DUP);
        const float w3 = row_bcast_dyn(p[(4 * h + 3) % NPL], ((4 * h + 3) / NPL) * DUP);
        p01[h] = pack2_bf16(w0, w1);
        p23[h] = pack2_bf16(w2, w3);
      }
      // dims 2k, 2k+1: (slot0, slot1) and (slot2, slot3) bf16 pairs via v_perm
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint32_t a0 = __builtin_amdgcn_perm(vf[1].w[k], vf[0].w[k], 0x05040100u);
        const uint32_t a1 = __builtin_amdgcn_perm(vf[1].w[k], vf[0].w[k], 0x07060302u);
        const uint32_t b0 = __builtin_amdgcn_perm(vf[3].w[k], vf[2].w[k], 0x05040100u);
        const uint32_t b1 = __builtin_amdgcn_perm(vf[3].w[k], vf[2].w[k], 0x07060302u);
#pragma unroll
        for (int h = 0; h < GW; ++h) {
          const bf16x2_t x01 = __builtin_bit_cast(bf16x2_t, p01[h]);
          const bf16x2_t x23 = __builtin_bit_cast(bf16x2_t, p23[h]);
          float t = __builtin_amdgcn_fdot2_f32_bf16(x01, __builtin_bit_cast(bf16x2_t, a0), acc[h][2 * k], false);
          acc[h][2 * k] = __builtin_amdgcn_fdot2_f32_bf16(x23, __builtin_bit_cast(bf16x2_t, b0), t, false);
          t = __builtin_amdgcn_fdot2_f32_bf16(x01, __builtin_bit_cast(bf16x2_t, a1), acc[h][2 * k + 1], false);
          acc[h][2 * k + 1] = __builtin_amdgcn_fdot2_f32_bf16(x23, __builtin_bit_cast(bf16x2_t, b1), t, false);
        }
      }
    } else {
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
  it.dirv = seq_direction(a.dir, a.cls, it.s);
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

template <int G, bool BF16>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(BF16 ? 4 : 1))) void decode_kernel(DecodeArgs a) {
  constexpr int GW = G > 4 ? 4 : G;     // heads per wave
  constexpr int HS = G / GW;            // waves sharing a block stream
  constexpr int NSTREAM = kWaves / HS;  // block streams per workgroup
  using LY = Layout<GW>;

  __shared__ int s_prefix[kMaxRowsLds + 1];
  __shared__ float s_acc[kWaves][GW][kHeadDim];
  __shared__ float s_m[kWaves][GW], s_l[kWaves][GW];
  __shared__ int s_scan[kThreads];
  __shared__ v4u_t s_q[kWaves][GW][16];   // bf16: each wave's query fragments, re-read per block

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

  Frag<BF16> q[GW];
  Frag<BF16> kf[4], vf[4];
  WaveState<GW, BF16> st;
  const bool primary = (C & (LY::DUP - 1)) == 0;
  const size_t lane_off = (size_t)R * kHeadDim + 8 * C;

  auto issue_k = [&](const Item& it, int i) -> int {
    const int blk = read_lane_i32(it.tbl, stream + NSTREAM * i);
    if (blk < 0 || blk >= a.num_blocks) return -1;
    const size_t base = ((size_t)blk * nkv + it.g) * kTileElems + lane_off;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      // With two waves per stream both read the same tile: keep it cacheable so
      // the second read is served on chip.
      if constexpr (HS == 1) kf[j].load_stream(a.k_pool, base + (size_t)(4 * j) * kHeadDim);
      else kf[j].load(a.k_pool, base + (size_t)(4 * j) * kHeadDim);
    }
    return blk;
  };
  auto issue_v = [&](const Item& it, int i) {
    const int blk = read_lane_i32(it.tbl, stream + NSTREAM * i);
    if (blk < 0 || blk >= a.num_blocks) return;
    const size_t base = ((size_t)blk * nkv + it.g) * kTileElems + lane_off;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if constexpr (HS == 1) vf[j].load_stream(a.v_pool, base + (size_t)(4 * j) * kHeadDim);
      else vf[j].load(a.v_pool, base + (size_t)(4 * j) * kHeadDim);
    }
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
    if constexpr (BF16) {   // park the query in LDS: its registers are free between blocks
      if (R == 0) {
#pragma unroll
        for (int h = 0; h < GW; ++h) s_q[w][h][C] = v4u_t{q[h].w[0], q[h].w[1], q[h].w[2], q[h].w[3]};
      }
    }
    st.reset();

    for (int i = 0; i < cur.nbw; ++i) {
      const int blk = blk_next;
      const int b = cur.b_begin + stream + NSTREAM * i;   // logical block index
      const bool more_here = i + 1 < cur.nbw;
      const bool more_next = !more_here && nxt_ok && nxt.nbw > 0;
      float sc[LY::NPL];
      if (blk >= 0) {
        if constexpr (BF16) {
          int cq = C;
          asm volatile("" : "+v"(cq));   // keeps the reads in the loop (not hoisted into registers)
#pragma unroll
          for (int h = 0; h < GW; ++h) {
            const v4u_t v = s_q[w][h][cq];
            q[h].w[0] = v.x; q[h].w[1] = v.y; q[h].w[2] = v.z; q[h].w[3] = v.w;
          }
        }
        st.scores(q, kf, a.scale_log2, C, sc);
      }
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
        store_out<BF16>(a.out, qh * kHeadDim + d, L > 0.0f ? A / L : 0.0f);
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
  c.dirv = seq_direction(a.dir, a.cls, c.s);
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

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

template <int G>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4))) void decode_mfma_kernel(DecodeArgs a) {
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
  v4u_t qf[4], kf[4], vf[4];
  floatx4_t acc[8];
  float m_ref = kNoMax, l_part = 0.0f;

  auto table = [&](const Cursor& c) -> int {
    const int blk = load_uniform(a.block_tables, (size_t)c.s * a.max_blocks_per_seq + c.b);
    return (blk >= 0 && blk < a.num_blocks) ? blk : -1;
  };
  auto issue_k = [&](int blk, int g) {
    if (blk < 0) return;
    const size_t base = ((size_t)blk * nkv + g) * kTileElems + k_lane;
#pragma unroll
    for (int c = 0; c < 4; ++c) kf[c] = load_nt(a.k_pool, base + 32 * c);
  };
  auto issue_v = [&](int blk, int g) {
    if (blk < 0) return;
    const size_t base = ((size_t)blk * nkv + g) * kTileElems + v_lane;
#pragma unroll
    for (int j = 0; j < 4; ++j) vf[j] = load_nt(a.v_pool, base + (size_t)j * kHeadDim);
  };
  auto load_q = [&](const Cursor& c) {
    const size_t qoff = ((size_t)c.row * Hq + c.g * G + col) * kHeadDim + 8 * grp;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      qf[k] = v4u_t{0u, 0u, 0u, 0u};
      if (head_lane) qf[k] = *reinterpret_cast<const v4u_t*>(static_cast<const uint16_t*>(a.q) + qoff + 32 * k);
    }
  };

  Cursor c0, c1;
  locate(a, s_pre, chunk, nch, t0, c0);
  int blk0 = table(c0);
  issue_k(blk0, c0.g);
  issue_v(blk0, c0.g);
  load_q(c0);
  bool whole = c0.b == 0;   // this wave saw the segment's first tile
  c1 = c0;
  int blk1 = -1;
  if (n > 1) {
    advance(a, c1);
    blk1 = table(c1);
  }
#pragma unroll
  for (int t = 0; t < 8; ++t) acc[t] = floatx4_t{0.0f, 0.0f, 0.0f, 0.0f};

  for (int i = 0; i < n; ++i) {
    // the tile after next: its table entry is read now, used one tile later
    Cursor c2 = c1;
    int blk2 = -1;
    if (i + 2 < n) {
      advance(a, c2);
      blk2 = table(c2);
    }
    floatx4_t sc = {0.0f, 0.0f, 0.0f, 0.0f};
    if (blk0 >= 0) {
#pragma unroll
      for (int k = 0; k < 4; ++k)
        sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kf[k]),
                                                     __builtin_bit_cast(bf16x8_t, qf[k]), sc, 0, 0, 0);
    }
    const bool seg_end = c0.b == c0.nblk - 1 || i + 1 == n;
    // K and query registers are free: the next tile's keys (and query on a new segment)
    if (i + 1 < n) {
      issue_k(blk1, c1.g);
      if (seg_end) load_q(c1);
    }
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
    // V registers are free: the next tile's values
    if (i + 1 < n) issue_v(blk1, c1.g);

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
    c0 = c1;
    blk0 = blk1;
    c1 = c2;
    blk1 = blk2;
  }
}

// Rows whose (row, KV head) segment was cut between workers: combine the
// partials o = sum_w 2^(m_w - M) acc_w / sum_w 2^(m_w - M) l_w. Rows without
// context get zeros; segments a single worker covered were written directly.
// One wave per (row, query head): lanes take 64 partials' (m, l) at a time,
// then every lane folds two head dims over the partials with eight loads in
// flight. (Merging inside the decode kernel instead would need device-scope
// release/acquire between workgroups, which on this chip writes back and
// invalidates a whole L2 per segment; the kernel boundary is far cheaper.)
constexpr int kMergeWaves = 4;

__global__ __launch_bounds__(kMergeWaves * kWave) void decode_mfma_merge_kernel(DecodeArgs a, int group) {
  const int lane = threadIdx.x & (kWave - 1);
  const int item = blockIdx.x * kMergeWaves + wave_id_uniform();
  if (item >= a.num_rows * a.num_q_heads) return;
  const int hq = item % a.num_q_heads;
  const int row = item / a.num_q_heads;
  const int g = hq / group, hl = hq - g * group;
  int s, ctx;
  resolve_row(a, row, s, ctx);
  uint32_t* out = reinterpret_cast<uint32_t*>(static_cast<uint16_t*>(a.out) + ((size_t)row * a.num_q_heads + hq) * kHeadDim) + lane;
  if (ctx <= 0) {
    *out = 0u;
    return;
  }
  const int nblk = (ctx + kBlockSize - 1) / kBlockSize;
  const int total = a.ws_rows[a.num_rows];
  const int workers = min(a.num_workers, total);
  const int64_t first_tile = (int64_t)a.ws_rows[row] + (int64_t)g * nblk;
  const int w0 = __builtin_amdgcn_readfirstlane(worker_of(first_tile, total, workers));
  const int w1 = __builtin_amdgcn_readfirstlane(worker_of(first_tile + nblk - 1, total, workers));
  if (w0 == w1) return;
  const size_t seg = (size_t)row * a.num_kv_heads + g;

  float M = kNoMax;
  for (int c = w0; c <= w1; c += kWave) {
    const int w = c + lane;
    if (w <= w1) M = fmaxf(M, a.ws_ml[2 * ((seg + w) * group + hl)]);
  }
  M = wave_max(M);
  float L = 0.0f, Ax = 0.0f, Ay = 0.0f;
  for (int c = w0; c <= w1; c += kWave) {
    const int w = c + lane;
    float wt = 0.0f;
    if (w <= w1) {
      const size_t slot = (seg + w) * group + hl;
      wt = fast_exp2(a.ws_ml[2 * slot] - M);
      L = fmaf(a.ws_ml[2 * slot + 1], wt, L);
    }
    const int cnt = min(kWave, w1 - c + 1);
    for (int j0 = 0; j0 < cnt; j0 += 8) {
      float2 v[8];
      float wj[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {   // indices clamped in range; padding gets weight 0
        const int j = min(j0 + u, cnt - 1);
        wj[u] = (j0 + u < cnt) ? __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wt), j)) : 0.0f;
        v[u] = reinterpret_cast<const float2*>(a.ws_acc + ((seg + c + j) * group + hl) * kHeadDim)[lane];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        Ax = fmaf(v[u].x, wj[u], Ax);
        Ay = fmaf(v[u].y, wj[u], Ay);
      }
    }
  }
  L = wave_sum(L);
  const float inv = L > 0.0f ? 1.0f / L : 0.0f;
  *out = pack2_bf16(Ax * inv, Ay * inv);
}

// Combine the split partials of every (row, head) whose context needed more
// than one split: o = sum_i 2^(m_i - M) acc_i / sum_i 2^(m_i - M) l_i.
template <bool BF16>
__global__ __launch_bounds__(kHeadDim) void decode_merge_kernel(DecodeArgs a) {
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
  store_out<BF16>(a.out, ((size_t)row * a.num_q_heads + hq) * kHeadDim + d, L > 0.0f ? A / L : 0.0f);
}

// Workgroups of `kernel` the device holds at once (queried once per device).
int resident_workgroups(const void* kernel, int slot) {
  constexpr int kMaxDevices = 64;
  constexpr int kSlots = 8;
  static int cache[kMaxDevices][kSlots];
  static std::mutex mu;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 1024;
  std::lock_guard<std::mutex> lock(mu);
  if (cache[dev][slot] == 0) {
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kThreads, 0) != hipSuccess || per_cu <= 0) per_cu = 4;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) cus = 256;
    cache[dev][slot] = per_cu * cus;
  }
  return cache[dev][slot];
}

// Workgroups of the bf16 decode grid at most (four workers each): what 256
// compute units hold at four waves per SIMD. The workspace is sized for it.
constexpr int kMaxDecodeGrid = 1024;

template <int G, bool BF16>
hipError_t launch_group(DecodeArgs a, hipStream_t stream, int slot) {
  if constexpr (BF16) {
    int grid = resident_workgroups(reinterpret_cast<const void*>(&decode_mfma_kernel<G>), slot);
    grid = grid < kMaxDecodeGrid ? grid : kMaxDecodeGrid;
    a.num_workers = grid * kWaves;
    hipLaunchKernelGGL((decode_mfma_kernel<G>), dim3(grid), dim3(kThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const unsigned merge_grid = (unsigned)(((long long)a.num_rows * a.num_q_heads + kMergeWaves - 1) / kMergeWaves);
    hipLaunchKernelGGL(decode_mfma_merge_kernel, dim3(merge_grid), dim3(kMergeWaves * kWave), 0, stream, a, G);
    return hipGetLastError();
  } else {
    const long long padded = (long long)a.num_rows * a.num_kv_heads * a.n_split_max;
    const int resident = resident_workgroups(reinterpret_cast<const void*>(&decode_kernel<G, false>), slot);
    const int grid = (int)(padded < resident ? padded : resident);
    if (grid <= 0) return hipSuccess;
    hipLaunchKernelGGL((decode_kernel<G, false>), dim3(grid), dim3(kThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.n_split_max <= 1) return e;
    hipLaunchKernelGGL((decode_merge_kernel<false>), dim3((unsigned)(a.num_rows * a.num_q_heads)),
                       dim3(kHeadDim), 0, stream, a);
    return hipGetLastError();
  }
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
           slots * 2 * sizeof(float);
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
    return;
  }
  a.ws_rows = nullptr;
  a.ws_acc = reinterpret_cast<float*>(base);
  a.ws_ml = base ? a.ws_acc + (size_t)a.num_rows * a.num_q_heads * a.n_split_max * kHeadDim : nullptr;
}

hipError_t launch_decode(DecodeArgs a, int group, bool bf16, hipStream_t stream) {
  switch (group * 2 + (bf16 ? 1 : 0)) {
    case 2: return launch_group<1, false>(a, stream, 0);
    case 3: return launch_group<1, true>(a, stream, 1);
    case 4: return launch_group<2, false>(a, stream, 2);
    case 5: return launch_group<2, true>(a, stream, 3);
    case 8: return launch_group<4, false>(a, stream, 4);
    case 9: return launch_group<4, true>(a, stream, 5);
    case 16: return launch_group<8, false>(a, stream, 6);
    case 17: return launch_group<8, true>(a, stream, 7);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace bros
