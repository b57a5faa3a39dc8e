// bros_attn_prefill_chunk (bf16) on gfx950 matrix cores.
//
// What it computes (Sec. 6: prefill rows of the mixed batch concatenated with a
// length table; chunked prefill on top of cached context, Sec. 2.2): row j of
// sequence s sits at position c0 + j, c0 = ctx - n, and attends to positions
// 0 .. c0 + j of the sequence, gathered from the bidirectional pool (Sec. 5.1).
//
// Tiling. A workgroup (4 waves) owns one (sequence, KV head, tile of QT
// positions) and all G = Hq / Hkv query heads of that KV head: 128 query rows,
// 32 per wave. Keys stream through LDS 64 at a time (four 16-slot blocks, one
// per wave), double-buffered: the next tile is fetched into registers while
// the current one is used, then staged into the other buffer. K is staged
// row-major [key][d] (272-byte rows), V transposed [d][key] (144-byte rows
// whose 8-byte key groups are XOR-swizzled by d / 8), which makes both the
// staging writes and the operand reads free of bank conflicts. The logical
// position of every staged key (or "invalid") sits beside them. Slots past
// the context or behind an invalid table entry are staged as zeros, so the
// matrix cores never see whatever the pool holds there.
//
// Both products run transposed, S^T = K Q^T and O^T += V^T P^T, with
// v_mfma_f32_32x32x16_bf16. In that orientation lane l owns query row l % 32:
// its 16 accumulator values of S^T are 16 keys of its own row, so the row
// max / sum need only one exchange between the two half-waves, the O rescale
// is lane-local, and the P operand of the second product is read straight out
// of the S accumulator (keys are permuted identically in P and V^T; the sum
// over keys does not care). The causal mask compares each key's logical
// position with the row's position, only on tiles that reach the diagonal or
// the context end: direction only reorders keys inside a block, which neither
// product sees. The running max moves lazily (only when a score exceeds it by
// more than 2^8), so the O rescale is rare.
#include "bros_device.h"
#include "bros_kernels.h"

#include <limits.h>
#include <math.h>

#include <type_traits>

namespace bros {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2_t;
typedef __attribute__((__vector_size__(2 * sizeof(float)))) float float2_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float floatx16;

constexpr int kThreads = 256;
constexpr int kKeys = 64;                          // keys per LDS tile (4 blocks)
constexpr int kKRow = kHeadDim * 2 + 16;           // bytes per staged K row (padded)
constexpr int kVRow = kKeys * 2 + 16;              // bytes per staged V^T row (padded)
constexpr int kRowsPerWave = 32;
constexpr float kRescaleSlack = 8.0f;              // log2 units
constexpr float kNoMax = -1.0e30f;
constexpr int kMaxTableLds = kPrefillMaxCtxMfma / kBlockSize;   // table entries staged in LDS

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }
__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {   // round to nearest even
  const float2_t f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}
// V^T layout: the 4-key group `chunk` (keys 4*chunk .. +3) of row d sits at
// byte d * kVRow + 8 * (chunk ^ (d / 8 % 16)).

template <int G>
__global__ __launch_bounds__(kThreads, 2) void prefill_mfma_kernel(PrefillArgs a) {
  constexpr int QT = 128 / G;   // positions per tile
  __shared__ __attribute__((aligned(16))) uint8_t s_k[2][kKeys * kKRow];
  __shared__ __attribute__((aligned(16))) uint8_t s_vt[2][kHeadDim * kVRow];
  __shared__ __attribute__((aligned(16))) int s_kpos[2][kKeys];
  __shared__ int s_blk_ok[2][4];   // the tile's four table entries were valid
  __shared__ int s_tbl[kMaxTableLds];

  // Work order. Consecutive workgroup ids land on different XCDs (id % 8),
  // each XCD with its own L2. When the number of (sequence, KV head) pairs is
  // a multiple of 8, pair p takes ids p, p + P, p + 2P, ... (P pairs), so all
  // its tiles run on XCD p % 8 and share that L2 for their K/V tiles, and
  // every XCD gets one pair of each group of 8 -- for the usual 8 KV heads,
  // one KV head of every sequence, which keeps the XCDs evenly loaded however
  // long the sequences are. Within a pair the longest rows come first.
  const int L = blockIdx.x;
  const int P = a.num_seqs * a.num_kv_heads;
  int pair, tile_rev;
  if ((P & 7) == 0) {
    pair = L % P;
    tile_rev = L / P;
  } else {
    pair = L / a.tiles_per_seq;
    tile_rev = L % a.tiles_per_seq;
  }
  const int g = pair % a.num_kv_heads;
  const int s = pair / a.num_kv_heads;
  const int tile = a.tiles_per_seq - 1 - tile_rev;

  const int q_begin = a.cu_q[s];
  const int n = a.cu_q[s + 1] - q_begin;
  const int t0 = tile * QT;
  if (q_begin < 0 || n <= 0 || q_begin + n > a.num_q_tokens || t0 >= n) return;
  const int c0 = a.ctx_lens[s] - n;
  if (c0 < 0) return;   // inconsistent lengths: rows left untouched
  const int ctx = min(a.ctx_lens[s], min(a.max_ctx, a.max_blocks_per_seq * kBlockSize));
  const int nblk = (ctx + kBlockSize - 1) / kBlockSize;
  const int dirv = seq_direction(a.dir, a.cls, s);
  const int rows_here = min(n, t0 + QT);
  const int kend = min(ctx, c0 + rows_here);
  const int n_tiles = (kend + kKeys - 1) / kKeys;
  // keys below this logical position are visible to every row of the workgroup
  const int full_below = min(ctx, c0 + t0 + 1);

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wv = wave_id_uniform();
  const int half = lane >> 5;
  const int mrow = lane & 31;
  const int r = kRowsPerWave * wv + mrow;
  const int head = g * G + r / QT;
  const int qrow = t0 + r % QT;
  const bool row_valid = qrow < n;
  const int qpos = row_valid ? c0 + qrow : -1;
  const int Hq = a.num_q_heads;

  // Q^T operand: for d-step c, lane holds Q[row][16c + 8*half .. +8).
  bf16x8_t qf[8];
  {
    const uint16_t* qp = static_cast<const uint16_t*>(a.q) + ((size_t)(q_begin + qrow) * Hq + head) * kHeadDim;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (row_valid) v = *reinterpret_cast<const uint4*>(qp + 16 * c + 8 * half);
      qf[c] = as_bf16x8(v);
    }
    // Consume the Q loads here: otherwise the first use inside the tile loop
    // waits for every outstanding load, including the prefetched tiles.
#pragma unroll
    for (int c = 0; c < 8; ++c) asm volatile("" : "+v"(qf[c]));
  }

  floatx16 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o[dt] = floatx16{};
  float m_run = kNoMax, l_run = 0.0f;

  const uint16_t* kpool = static_cast<const uint16_t*>(a.k_pool);
  const uint16_t* vpool = static_cast<const uint16_t*>(a.v_pool);
  // Staging: wave u copies block u of the tile; lane (sq, dc) copies slots
  // 4sq .. 4sq+3 and head dims [8dc, 8dc+8) of its K and V tiles.
  const int sq = lane >> 4;
  const int dc = lane & 15;
  // V^T staging: rows 8dc .. 8dc+7, key group (4wv + sq) swizzled by dc
  const int vt_write_base = 8 * dc * kVRow + ((((4 * wv + sq) ^ dc) & 15) << 3);
  // V^T operand reads: row d = 32dt + mrow, group 4c2 + 2hi + half; the
  // swizzle (d/8 = 4dt + mrow/8) splits into a per-lane low part and a
  // compile-time high part: group ^ swz = 4 (c2 ^ dt) + ((2hi + half) ^ (mrow/8 % 4)).
  const int swz_lo = (mrow >> 3) & 3;
  const int vt_read_lo = mrow * kVRow + ((half ^ swz_lo) << 3);
  const int vt_read_hi = mrow * kVRow + (((2 + half) ^ swz_lo) << 3);

  // The sequence's table entries for this chunk, staged once in LDS, so a
  // table lookup never adds a global load inside the tile loop.
  // (The host sends contexts longer than kMaxTableLds blocks to the vector
  // path, so the whole table of the sequence fits.)
  const int nblk_tbl = min(nblk, kMaxTableLds);
  for (int i = tid; i < nblk_tbl; i += kThreads) s_tbl[i] = a.block_tables[(size_t)s * a.max_blocks_per_seq + i];
  __syncthreads();
  auto table = [&](int b) -> int {
    const int blk = b < nblk_tbl ? s_tbl[b] : -1;
    return (blk >= 0 && blk < a.num_blocks) ? blk : -1;
  };

  // Two register sets (A, B): tile kt + 2 is requested while tile kt is
  // computed. Every fetch issues exactly eight loads (an invalid block reads
  // block 0 and is zeroed when staged), so the waits before staging only
  // cover the older set.
  uint4 kA[4], vA[4], kB[4], vB[4];
  int blkA = -1, blkB = -1;
  auto fetch = [&](int kt, auto set) __attribute__((always_inline)) {
    constexpr int SET = decltype(set)::value;
    uint4(&kr)[4] = SET == 0 ? kA : kB;
    uint4(&vr)[4] = SET == 0 ? vA : vB;
    const int blk = table(kt * 4 + wv);
    if constexpr (SET == 0) blkA = blk; else blkB = blk;
    const size_t base = (((size_t)max(blk, 0) * a.num_kv_heads + g) * kBlockSize + 4 * sq) * kHeadDim + 8 * dc;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      kr[j] = *reinterpret_cast<const uint4*>(kpool + base + j * kHeadDim);
      vr[j] = *reinterpret_cast<const uint4*>(vpool + base + j * kHeadDim);
    }
  };
  auto stage = [&](int buf, int kt, auto set) __attribute__((always_inline)) {
    constexpr int SET = decltype(set)::value;
    uint4(&kr)[4] = SET == 0 ? kA : kB;
    uint4(&vr)[4] = SET == 0 ? vA : vB;
    const int blk = SET == 0 ? blkA : blkB;
    const int b = kt * 4 + wv;
    const int key0 = 16 * wv + 4 * sq;
    if (!(blk >= 0 && (b + 1) * kBlockSize <= ctx)) {   // tail or invalid block: zero what is not context
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (!(blk >= 0 && b * kBlockSize + slot_of_offset(4 * sq + j, dirv) < ctx)) {
          kr[j] = make_uint4(0, 0, 0, 0);
          vr[j] = kr[j];
        }
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
      *reinterpret_cast<uint4*>(s_k[buf] + (key0 + j) * kKRow + dc * 16) = kr[j];
    // V^T: dims 2k and 2k+1 of the four slots, as two 8-byte key groups
    const uint32_t w0[4] = {vr[0].x, vr[0].y, vr[0].z, vr[0].w};
    const uint32_t w1[4] = {vr[1].x, vr[1].y, vr[1].z, vr[1].w};
    const uint32_t w2[4] = {vr[2].x, vr[2].y, vr[2].z, vr[2].w};
    const uint32_t w3[4] = {vr[3].x, vr[3].y, vr[3].z, vr[3].w};
    // rows d = 8dc + 2k (+1) all have d / 8 = dc, so the swizzled group is
    // the same for the eight rows this lane writes
    uint8_t* vt_lane = s_vt[buf] + vt_write_base;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      uint2 lo, hi;
      lo.x = __builtin_amdgcn_perm(w1[k], w0[k], 0x05040100u);
      lo.y = __builtin_amdgcn_perm(w3[k], w2[k], 0x05040100u);
      hi.x = __builtin_amdgcn_perm(w1[k], w0[k], 0x07060302u);
      hi.y = __builtin_amdgcn_perm(w3[k], w2[k], 0x07060302u);
      *reinterpret_cast<uint2*>(vt_lane + (2 * k) * kVRow) = lo;
      *reinterpret_cast<uint2*>(vt_lane + (2 * k + 1) * kVRow) = hi;
    }
    if (dc == 0) {
      int kp[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int pos = b * kBlockSize + slot_of_offset(4 * sq + j, dirv);
        kp[j] = (blk >= 0 && pos < ctx) ? pos : INT_MAX;
      }
      *reinterpret_cast<int4*>(&s_kpos[buf][key0]) = make_int4(kp[0], kp[1], kp[2], kp[3]);
    }
    if (lane == 0) s_blk_ok[buf][wv] = blk >= 0;
  };

  auto compute = [&](int kt) __attribute__((always_inline)) {
    const int buf = kt & 1;
    const uint8_t* sk = s_k[buf];
    const uint8_t* svt = s_vt[buf];
    const int* skpos = s_kpos[buf];

    // S^T = K Q^T for keys [32*st, 32*st + 32).
    floatx16 sacc[2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      sacc[st] = floatx16{};
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const uint4 kv = *reinterpret_cast<const uint4*>(sk + (32 * st + mrow) * kKRow + (16 * c + 8 * half) * 2);
        sacc[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kv), qf[c], sacc[st], 0, 0, 0);
      }
    }

    // Scale to log2 units; mask by logical position where the tile needs it.
    // Accumulator j of sub-tile st is key 32*st + 8*(j/4) + 4*half + j%4.
    const bool full = (kt + 1) * kKeys <= full_below && s_blk_ok[buf][0] && s_blk_ok[buf][1] &&
                      s_blk_ok[buf][2] && s_blk_ok[buf][3];
    float mraw = -INFINITY;   // max of the raw scores (scale > 0 commutes with max)
    if (full) {
#pragma unroll
      for (int st = 0; st < 2; ++st) {
#pragma unroll
        for (int j = 0; j < 16; ++j) mraw = fmaxf(mraw, sacc[st][j]);
      }
    } else {
#pragma unroll
      for (int st = 0; st < 2; ++st) {
#pragma unroll
        for (int jq = 0; jq < 4; ++jq) {
          const int4 kp4 = *reinterpret_cast<const int4*>(skpos + 32 * st + 8 * jq + 4 * half);
          const int kpv[4] = {kp4.x, kp4.y, kp4.z, kp4.w};
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            const int j = 4 * jq + jj;
            const float v = kpv[jj] <= qpos ? sacc[st][j] : -INFINITY;
            sacc[st][j] = v;
            mraw = fmaxf(mraw, v);
          }
        }
      }
    }
    mraw = fmaxf(mraw, __shfl_xor(mraw, 32));
    const float mx = mraw * a.scale_log2;   // log2 units; -inf when nothing is visible
    if (__builtin_amdgcn_ballot_w64(mx > m_run + kRescaleSlack) != 0) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = fast_exp2(m_run - m_new);
      l_run *= alpha;
      m_run = m_new;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
        for (int j = 0; j < 16; ++j) o[dt][j] *= alpha;
      }
    }
    float psum = 0.0f;
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const float p = fast_exp2(fmaf(sacc[st][j], a.scale_log2, -m_run));
        sacc[st][j] = p;
        psum += p;
      }
    }
    l_run += psum;

    // P^T operand for key step c2 (16 keys): accumulators 8*(c2%2) .. +8 of sub-tile c2/2.
    bf16x8_t pf[4];
#pragma unroll
    for (int c2 = 0; c2 < 4; ++c2) {
      const floatx16& sv = sacc[c2 >> 1];
      const int j0 = 8 * (c2 & 1);
      uint4 pk;
      pk.x = pack2_bf16(sv[j0 + 0], sv[j0 + 1]);
      pk.y = pack2_bf16(sv[j0 + 2], sv[j0 + 3]);
      pk.z = pack2_bf16(sv[j0 + 4], sv[j0 + 5]);
      pk.w = pack2_bf16(sv[j0 + 6], sv[j0 + 7]);
      pf[c2] = as_bf16x8(pk);
    }

    // O^T += V^T P^T: V^T operand row d holds keys 16c2 + 4*half + {0..3} and
    // 16c2 + 8 + 4*half + {0..3}, the same permutation the P operand carries.
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
      for (int c2 = 0; c2 < 4; ++c2) {
        const int cst = 32 * dt * kVRow + 32 * (c2 ^ dt);
        const uint2 lo = *reinterpret_cast<const uint2*>(svt + vt_read_lo + cst);
        const uint2 hi = *reinterpret_cast<const uint2*>(svt + vt_read_hi + cst);
        const uint4 vv = make_uint4(lo.x, lo.y, hi.x, hi.y);
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vv), pf[c2], o[dt], 0, 0, 0);
      }
    }
  };

  // Tile kt is computed from buffer kt % 2 while tile kt + 1 (already in
  // registers) is staged into the other buffer, which was last read before
  // the previous barrier; tile kt + 2 is requested before the computing starts.
  using SetA = std::integral_constant<int, 0>;
  using SetB = std::integral_constant<int, 1>;
  // Fetches and stages run unconditionally (a tile past the end reads block 0
  // and stages zeros into the buffer nobody reads next), so every iteration
  // issues the same loads and the waits stay exact; only compute is guarded.
  fetch(0, SetA{});
  fetch(1, SetB{});
  stage(0, 0, SetA{});
  __syncthreads();
  for (int kt = 0; kt < n_tiles; kt += 2) {
    fetch(kt + 2, SetA{});
    compute(kt);
    stage(1, kt + 1, SetB{});
    __syncthreads();
    fetch(kt + 3, SetB{});
    if (kt + 1 < n_tiles) compute(kt + 1);
    stage(0, kt + 2, SetA{});
    __syncthreads();
  }

  // Each half-wave summed its own keys; the row total is their sum.
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (row_valid) {
    const float inv = l_tot > 0.0f ? 1.0f / l_tot : 0.0f;
    uint16_t* op = static_cast<uint16_t*>(a.out) + ((size_t)(q_begin + qrow) * Hq + head) * kHeadDim;
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

}  // namespace

int prefill_positions_per_tile(int group) { return 128 / group; }

hipError_t launch_prefill_mfma(const PrefillArgs& a, int group, int num_tiles_total, hipStream_t stream) {
  if (num_tiles_total <= 0) return hipSuccess;
  switch (group) {
    case 1: hipLaunchKernelGGL(prefill_mfma_kernel<1>, dim3(num_tiles_total), dim3(kThreads), 0, stream, a); break;
    case 2: hipLaunchKernelGGL(prefill_mfma_kernel<2>, dim3(num_tiles_total), dim3(kThreads), 0, stream, a); break;
    case 4: hipLaunchKernelGGL(prefill_mfma_kernel<4>, dim3(num_tiles_total), dim3(kThreads), 0, stream, a); break;
    case 8: hipLaunchKernelGGL(prefill_mfma_kernel<8>, dim3(num_tiles_total), dim3(kThreads), 0, stream, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace bros
