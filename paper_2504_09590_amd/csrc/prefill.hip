// bros_attn_prefill_chunk (bf16) on gfx950 matrix cores.
//
// What it computes (Sec. 6: prefill rows of the mixed batch concatenated with a
// length table; chunked prefill on top of cached context, Sec. 2.2): row j of
// sequence s sits at position c0 + j, c0 = ctx - n, and attends to positions
// 0 .. c0 + j of the sequence, gathered from the bidirectional pool (Sec. 5.1).
//
// Tiling. A workgroup (4 waves) owns one (sequence, KV head, tile of QT
// positions) and all G = Hq / Hkv query heads of that KV head: 128 query rows,
// 32 per wave. Keys stream through LDS 64 at a time (four 16-slot blocks):
// K is staged row-major [key][d], V transposed [d][key], and the logical
// position of every staged key (or "invalid") beside them. Slots past the
// context or behind an invalid table entry are staged as zeros, so the
// matrix cores never see whatever the pool holds there.
//
// Both products run transposed, S^T = K Q^T and O^T += V^T P^T, with
// v_mfma_f32_32x32x16_bf16. In that orientation lane l owns query row l % 32:
// its 16 accumulator values of S^T are 16 keys of its own row, so the row
// max / sum need only one exchange between the two half-waves, the O rescale
// is lane-local, and the P operand of the second product is read straight out
// of the S accumulator (keys are permuted identically in P and V^T; the sum
// over keys does not care). The causal mask compares each key's logical
// position with the row's position: direction only reorders keys inside a
// block, which neither product sees.
#include "bros_device.h"
#include "bros_kernels.h"

#include <limits.h>
#include <math.h>

namespace bros {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float floatx16;

constexpr int kThreads = 256;
constexpr int kKeys = 64;                          // keys per LDS tile (4 blocks)
constexpr int kKRow = kHeadDim * 2 + 16;           // bytes per staged K row (padded)
constexpr int kVRow = kKeys * 2 + 8;               // bytes per staged V^T row (padded)
constexpr int kRowsPerWave = 32;

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

template <int G>
__global__ __launch_bounds__(kThreads) void prefill_mfma_kernel(PrefillArgs a) {
  constexpr int QT = 128 / G;   // positions per tile
  // Two LDS buffers: tile kt is read from buffer kt % 2 while tile kt + 1,
  // already fetched into registers, is staged into the other one.
  __shared__ __attribute__((aligned(16))) uint8_t s_k[2][kKeys * kKRow];
  __shared__ __attribute__((aligned(16))) uint8_t s_vt[2][kHeadDim * kVRow];
  __shared__ __attribute__((aligned(16))) int s_kpos[2][kKeys];

  // XCD-aware order: consecutive workgroup ids land on different XCDs (id % 8),
  // so give each XCD a contiguous run of work items. The tiles of one
  // (sequence, KV head) then share that XCD's L2 for their K/V tiles.
  const int T = gridDim.x;
  const int L = blockIdx.x;
  const int xcd = L & 7, per = T >> 3, rem = T & 7;
  const int work = xcd * per + min(xcd, rem) + (L >> 3);
  const int tile_rev = work % a.tiles_per_seq;
  const int rest = work / a.tiles_per_seq;
  const int g = rest % a.num_kv_heads;
  const int s = rest / a.num_kv_heads;
  const int tile = a.tiles_per_seq - 1 - tile_rev;   // longest rows first

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
  }

  floatx16 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o[dt] = floatx16{};
  float m_run = -INFINITY, l_run = 0.0f;

  const uint16_t* kpool = static_cast<const uint16_t*>(a.k_pool);
  const uint16_t* vpool = static_cast<const uint16_t*>(a.v_pool);
  const int slot = tid >> 4;   // staging: thread copies slot `slot`, dims [8*dc, 8*dc+8) of each block
  const int dc = tid & 15;

  // Global -> registers for tile kt: thread copies slot `slot`, dims
  // [8*dc, 8*dc+8) of each of the tile's four blocks (each block's tile is
  // 4 KiB contiguous, so a wave's load instruction reads 1 KiB contiguous).
  uint4 kreg[4], vreg[4];
  int kp[4];
  auto fetch = [&](int kt) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int b = kt * 4 + u;
      int blk = -1;
      if (b < nblk) blk = a.block_tables[(size_t)s * a.max_blocks_per_seq + b];
      const int pos = b * kBlockSize + slot_of_offset(slot, dirv);
      const bool valid = blk >= 0 && blk < a.num_blocks && pos < ctx;
      kreg[u] = make_uint4(0, 0, 0, 0);
      vreg[u] = kreg[u];
      if (valid) {
        const size_t off = (((size_t)blk * a.num_kv_heads + g) * kBlockSize + slot) * kHeadDim + 8 * dc;
        kreg[u] = *reinterpret_cast<const uint4*>(kpool + off);
        vreg[u] = *reinterpret_cast<const uint4*>(vpool + off);
      }
      kp[u] = valid ? pos : INT_MAX;
    }
  };
  // Registers -> LDS buffer `buf`: K row-major, V transposed, key positions.
  auto stage = [&](int buf) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int key = u * kBlockSize + slot;
      *reinterpret_cast<uint4*>(s_k[buf] + key * kKRow + dc * 16) = kreg[u];
      const uint32_t w4[4] = {vreg[u].x, vreg[u].y, vreg[u].z, vreg[u].w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint16_t val = (uint16_t)((e & 1) ? (w4[e >> 1] >> 16) : (w4[e >> 1] & 0xffffu));
        *reinterpret_cast<uint16_t*>(s_vt[buf] + (8 * dc + e) * kVRow + key * 2) = val;
      }
      if (dc == 0) s_kpos[buf][key] = kp[u];
    }
  };

  if (n_tiles > 0) {
    fetch(0);
    stage(0);
  }
  __syncthreads();

  for (int kt = 0; kt < n_tiles; ++kt) {
    const int buf = kt & 1;
    const bool more = kt + 1 < n_tiles;
    if (more) fetch(kt + 1);   // in flight while this tile is computed
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

    // Causal / validity mask by logical position, then the online softmax.
    // Accumulator j of sub-tile st is key 32*st + 8*(j/4) + 4*half + j%4.
    float mx = -INFINITY;
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        const int4 kp4 = *reinterpret_cast<const int4*>(skpos + 32 * st + 8 * jq + 4 * half);
        const int kpv[4] = {kp4.x, kp4.y, kp4.z, kp4.w};
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const int j = 4 * jq + jj;
          const float v = kpv[jj] <= qpos ? sacc[st][j] * a.scale_log2 : -INFINITY;
          sacc[st][j] = v;
          mx = fmaxf(mx, v);
        }
      }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mnew = fmaxf(m_run, mx);
    const float mu = mnew == -INFINITY ? 0.0f : mnew;
    const float alpha = fast_exp2(m_run - mu);
    float psum = 0.0f;
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const float p = fast_exp2(sacc[st][j] - mu);
        sacc[st][j] = p;
        psum += p;
      }
    }
    l_run = fmaf(l_run, alpha, psum);
    m_run = mnew;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
      for (int j = 0; j < 16; ++j) o[dt][j] *= alpha;
    }

    // P^T operand for key step c2 (16 keys): accumulators 8*(c2%2) .. +8 of sub-tile c2/2.
    bf16x8_t pf[4];
#pragma unroll
    for (int c2 = 0; c2 < 4; ++c2) {
      uint4 pk;
      pk.x = pack_bf16x2(sacc[c2 >> 1][8 * (c2 & 1) + 0], sacc[c2 >> 1][8 * (c2 & 1) + 1]);
      pk.y = pack_bf16x2(sacc[c2 >> 1][8 * (c2 & 1) + 2], sacc[c2 >> 1][8 * (c2 & 1) + 3]);
      pk.z = pack_bf16x2(sacc[c2 >> 1][8 * (c2 & 1) + 4], sacc[c2 >> 1][8 * (c2 & 1) + 5]);
      pk.w = pack_bf16x2(sacc[c2 >> 1][8 * (c2 & 1) + 6], sacc[c2 >> 1][8 * (c2 & 1) + 7]);
      pf[c2] = as_bf16x8(pk);
    }

    // O^T += V^T P^T: V^T operand row d holds keys 16c2 + 4*half + {0..3} and
    // 16c2 + 8 + 4*half + {0..3}, the same permutation the P operand carries.
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const uint8_t* vrow = svt + (32 * dt + mrow) * kVRow;
#pragma unroll
      for (int c2 = 0; c2 < 4; ++c2) {
        const uint2 lo = *reinterpret_cast<const uint2*>(vrow + (16 * c2 + 4 * half) * 2);
        const uint2 hi = *reinterpret_cast<const uint2*>(vrow + (16 * c2 + 8 + 4 * half) * 2);
        const uint4 vv = make_uint4(lo.x, lo.y, hi.x, hi.y);
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vv), pf[c2], o[dt], 0, 0, 0);
      }
    }
    // The other buffer was last read in the previous iteration, before the
    // barrier that ended it, so it can be overwritten now.
    if (more) stage(buf ^ 1);
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
        w.x = pack_bf16x2(o[dt][4 * jq + 0] * inv, o[dt][4 * jq + 1] * inv);
        w.y = pack_bf16x2(o[dt][4 * jq + 2] * inv, o[dt][4 * jq + 3] * inv);
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
