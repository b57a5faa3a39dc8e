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
// per wave), double-buffered. The pool's K and V rows go straight from global
// memory into LDS (global_load_lds, no registers, no vector ALU), both
// row-major [key][d] with the 16-byte chunks of row r permuted by
// chunk ^ swz(r); the V^T operand is read with the transposing LDS load
// (ds_read_b64_tr_b16). With that permutation the K operand reads and the
// transposing V reads are both free of bank conflicts. The logical position
// of every key (or "invalid") sits beside them. V rows of slots past the
// context or behind an invalid table entry are overwritten with zeros once
// their load has landed, so the matrix cores never multiply whatever the
// pool holds there (K rows there only produce scores that are masked).
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
constexpr int kRowBytes = kHeadDim * 2;           // bytes of one K or V row
constexpr int kTileBytes = kKeys * kRowBytes;      // one K or V tile in LDS
constexpr int kRowsPerWave = 32;
constexpr float kRescaleSlack = 8.0f;              // log2 units
constexpr float kNoMax = -1.0e30f;
constexpr int kMaxTableLds = kPrefillMaxCtxMfma / kBlockSize;   // table entries staged in LDS

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }
__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {   // round to nearest even
  const float2_t f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}
// 16-byte chunk c of row r of a K or V tile sits at byte r * 256 + 16 * (c ^ swz(r)).
__device__ __forceinline__ int swz(int r) { return ((r & 7) << 1) | ((r >> 3) & 1); }

typedef short v4s_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint2 lds_read_tr(const uint8_t* p) {   // ds_read_b64_tr_b16
  const v4s_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (v4s_t __attribute__((address_space(3)))*)(p));
  return __builtin_bit_cast(uint2, v);
}
__device__ __forceinline__ void load_to_lds(const uint16_t* src, uint8_t* dst) {   // 16 bytes per lane at dst + 16 * lane
  __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                   (__attribute__((address_space(3))) void*)dst, 16, 0, 0);
}
// Workgroup barrier for the tile pipeline: this wave's LDS reads and writes
// are complete (lgkmcnt 0) and the compiler may not move memory accesses
// across it. Loads into LDS still in flight (the tile two ahead) are not
// waited for -- a fence would wait for them -- so the wave that issued a tile
// waits for it explicitly (wait_vmem) before the barrier that publishes it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}
// s_waitcnt with only the vector-memory count limited (expcnt and lgkmcnt at maximum).
template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 16, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0F70 | N);
}

template <int G>
__global__ __launch_bounds__(kThreads, 2) void prefill_mfma_kernel(PrefillArgs a) {
  constexpr int QT = 128 / G;   // positions per tile
  // one array per buffer, so the compiler sees that reads of one buffer do not
  // alias the loads in flight into the other
  __shared__ __attribute__((aligned(1024))) uint8_t s_k0[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t s_k1[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t s_v0[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t s_v1[kTileBytes];
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
  // Loads: wave wv brings block wv of the tile, rows 16wv .. 16wv + 15; load i
  // covers rows 16wv + 4i + lane / 16, lane writing physical chunk lane % 16,
  // which holds logical chunk (lane % 16) ^ swz(row).
  const int ld_slot = lane >> 4;
  // K operand (S^T = K Q^T, d-step c): row 32st + mrow, logical chunk 2c + half.
  const int k_sw = swz(mrow);
  const int k_lane = mrow * kRowBytes + (((half ^ k_sw) & 1) << 4);
  // V^T operand via the transposing read, per (dt, part): lane (group j = lane /
  // 16, q = lane % 4, t = lane % 16 / 4) reads dims 32dt + 16(j % 2) + 4q ..+3 of
  // key 16c2 + 8part + 4half + t (key order shared with the P operand).
  const int tr_j = lane >> 4, tr_q = lane & 3, tr_t = (lane >> 2) & 3;
  int v_off[2];   // per part, without the dt-dependent chunk bits
  int v_sw[2];
#pragma unroll
  for (int part = 0; part < 2; ++part) {
    const int key = 8 * part + 4 * half + tr_t;   // mod 16; + 16c2 is a row offset
    v_sw[part] = swz(key);
    v_off[part] = key * kRowBytes + ((((2 * (tr_j & 1) + (tr_q >> 1)) ^ v_sw[part]) & 3) << 4) + (tr_q & 1) * 8;
  }

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

  // Tile kt into buffer `buf`: eight 1 KiB loads per wave, always issued (a
  // tile past the end reads block 0 and is marked invalid), so the wait for the
  // older tile is an exact count.
  auto load_tile = [&](int kt, auto bufc) __attribute__((always_inline)) {
    constexpr int BUF = decltype(bufc)::value;
    uint8_t* dk = BUF == 0 ? s_k0 : s_k1;
    uint8_t* dv = BUF == 0 ? s_v0 : s_v1;
    const int blk = table(kt * 4 + wv);
    const size_t base = ((size_t)max(blk, 0) * a.num_kv_heads + g) * kBlockSize * kHeadDim;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 16 * wv + 4 * i + ld_slot;
      const size_t src = base + (size_t)(4 * i + ld_slot) * kHeadDim + (size_t)(((lane & 15) ^ swz(row)) << 3);
      load_to_lds(kpool + src, dk + (16 * wv + 4 * i) * kRowBytes);
      load_to_lds(vpool + src, dv + (16 * wv + 4 * i) * kRowBytes);
    }
  };
  // Once this wave's loads of tile kt have landed: zero the V rows of slots
  // that are not context, record key positions and block validity.
  auto fixup = [&](int kt, auto bufc) __attribute__((always_inline)) {
    constexpr int BUF = decltype(bufc)::value;
    uint8_t* dv = BUF == 0 ? s_v0 : s_v1;
    const int b = kt * 4 + wv;
    const int blk = table(b);
    if (!(blk >= 0 && (b + 1) * kBlockSize <= ctx)) {   // tail or invalid block
#pragma unroll
      for (int p4 = 0; p4 < 4; ++p4) {
        const int slot = 4 * p4 + ld_slot;
        if (!(blk >= 0 && b * kBlockSize + slot_of_offset(slot, dirv) < ctx))
          *reinterpret_cast<uint4*>(dv + (16 * wv + slot) * kRowBytes + (lane & 15) * 16) = make_uint4(0, 0, 0, 0);
      }
    }
    if (lane < kBlockSize) {
      const int pos = b * kBlockSize + slot_of_offset(lane, dirv);
      s_kpos[BUF][16 * wv + lane] = (blk >= 0 && pos < ctx) ? pos : INT_MAX;
    }
    if (lane == 0) s_blk_ok[BUF][wv] = blk >= 0;
  };

  auto compute = [&](int kt, auto bufc) __attribute__((always_inline)) {
    constexpr int buf = decltype(bufc)::value;
    const uint8_t* sk = buf == 0 ? s_k0 : s_k1;
    const uint8_t* sv = buf == 0 ? s_v0 : s_v1;
    const int* skpos = s_kpos[buf];

    // S^T = K Q^T for keys [32*st, 32*st + 32).
    floatx16 sacc[2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      sacc[st] = floatx16{};
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        // logical chunk 2c + half of row 32st + mrow (swz(32st + mrow) = swz(mrow))
        const uint4 kv = *reinterpret_cast<const uint4*>(sk + 32 * st * kRowBytes + k_lane + (((2 * c) ^ (k_sw & 14)) << 4));
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
      // chunk 4dt + (2(j % 2) + q / 2) of the row: the dt bits XOR the swizzle's high bits
      const int off0 = v_off[0] + (((4 * dt) ^ (v_sw[0] & 12)) << 4);
      const int off1 = v_off[1] + (((4 * dt) ^ (v_sw[1] & 12)) << 4);
#pragma unroll
      for (int c2 = 0; c2 < 4; ++c2) {
        const uint2 lo = lds_read_tr(sv + 16 * c2 * kRowBytes + off0);
        const uint2 hi = lds_read_tr(sv + 16 * c2 * kRowBytes + off1);
        const uint4 vv = make_uint4(lo.x, lo.y, hi.x, hi.y);
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vv), pf[c2], o[dt], 0, 0, 0);
      }
    }
  };

  // Tile kt is computed from buffer kt % 2 while tile kt + 1 lands in the
  // other; after the barrier that frees a buffer, the tile two ahead is
  // requested into it, then this wave waits for its own loads of the next tile
  // (every older load: eight per tile are younger), fixes it up, and a second
  // barrier publishes it.
  using Buf0 = std::integral_constant<int, 0>;
  using Buf1 = std::integral_constant<int, 1>;
  load_tile(0, Buf0{});
  load_tile(1, Buf1{});
  wait_vmem<8>();
  fixup(0, Buf0{});
  lds_barrier();
  for (int kt = 0; kt < n_tiles; kt += 2) {
    compute(kt, Buf0{});
    lds_barrier();
    load_tile(kt + 2, Buf0{});
    wait_vmem<8>();
    fixup(kt + 1, Buf1{});
    lds_barrier();
    if (kt + 1 < n_tiles) compute(kt + 1, Buf1{});
    lds_barrier();
    load_tile(kt + 3, Buf1{});
    wait_vmem<8>();
    fixup(kt + 2, Buf0{});
    lds_barrier();
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
