// bros_attn_decode on gfx950: split-K paged attention over the bidirectional pool.
//
// What it computes (Sec. 2.1 decode attention over the cached KV; Sec. 5.1
// bidirectional slot order; Sec. 6 direction-aware paged kernel): for query
// row r of sequence s and query head h in KV group g = h / G,
//     out[r][h] = sum_p softmax_p(scale * q[r][h] . K[p][g]) V[p][g],  p < ctx(r).
//
// Work decomposition: one workgroup per (row, KV head, split of up to
// `split_blocks` blocks); its four waves take every fourth block of the split.
// A (block, KV head) tile is 16 slots x 128 head dims, contiguous in the pool
// ([num_blocks][Hkv][16][128]), so each load instruction of a wave reads 1 KiB
// contiguous. Lane (R = lane / 16, C = lane % 16) holds slots R, R+4, R+8,
// R+12 and head dims [8C, 8C+8) of the K and V tiles; the G query heads of the
// group reuse every loaded tile (GQA sharing).
//
// Softmax. Direction only decides which physical slots hold valid positions:
// attention is a sum over the set of cached tokens, so each score is paired
// with the V row of the same physical slot and the logical position
// b*16 + (dir > 0 ? slot : 15 - slot) is only compared with the context
// length (tail block). Invalid slots are removed by selection, never by
// multiplication, so whatever they hold (a peer request's tokens, NaNs) cannot
// leak. Each 16-lane row keeps its own online-softmax state in log2 units;
// rows, then waves, then splits are merged with the usual max-rescaling.
#include "bros_device.h"
#include "bros_kernels.h"

#include <math.h>

namespace bros {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kTileElems = kBlockSize * kHeadDim;   // one (block, KV head) tile

typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2_t;

// Eight consecutive head-dim elements of one slot (or of one query row).
template <bool BF16> struct Frag;
template <> struct Frag<true> {
  uint4 w;
  __device__ void load(const void* base, size_t elem) { w = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + elem); }
  __device__ void zero() { w = make_uint4(0, 0, 0, 0); }
  __device__ float at(int e) const {
    const uint32_t x = (e >> 1) == 0 ? w.x : (e >> 1) == 1 ? w.y : (e >> 1) == 2 ? w.z : w.w;
    return (e & 1) ? bf16_hi(x) : bf16_lo(x);
  }
  __device__ float dot(const Frag& k) const {   // products are exact, one rounding per pair
    float acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w.x), __builtin_bit_cast(bf16x2_t, k.w.x), 0.0f, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w.y), __builtin_bit_cast(bf16x2_t, k.w.y), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w.z), __builtin_bit_cast(bf16x2_t, k.w.z), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w.w), __builtin_bit_cast(bf16x2_t, k.w.w), acc, false);
    return acc;
  }
};
template <> struct Frag<false> {
  float4 a, b;
  __device__ void load(const void* base, size_t elem) {
    const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(base) + elem);
    a = p[0];
    b = p[1];
  }
  __device__ void zero() { a = make_float4(0, 0, 0, 0); b = a; }
  __device__ float at(int e) const {
    const float4& v = e < 4 ? a : b;
    const int i = e & 3;
    return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
  }
  __device__ float dot(const Frag& k) const {
    float acc = a.x * k.a.x;
    acc = fmaf(a.y, k.a.y, acc);
    acc = fmaf(a.z, k.a.z, acc);
    acc = fmaf(a.w, k.a.w, acc);
    acc = fmaf(b.x, k.b.x, acc);
    acc = fmaf(b.y, k.b.y, acc);
    acc = fmaf(b.z, k.b.z, acc);
    acc = fmaf(b.w, k.b.w, acc);
    return acc;
  }
};

template <bool BF16>
__device__ __forceinline__ void store_out(void* out, size_t elem, float v) {
  if constexpr (BF16) static_cast<uint16_t*>(out)[elem] = (uint16_t)f32_to_bf16_bits(v);
  else static_cast<float*>(out)[elem] = v;
}

// Resolve query row -> (sequence, visible context). Shared by both kernels.
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

template <int G, bool BF16>
__global__ __launch_bounds__(kThreads) void decode_split_kernel(DecodeArgs a) {
  const int SB = a.split_blocks;
  const int nkv = a.num_kv_heads;
  const int lin = blockIdx.x;
  const int split = lin % a.n_split_max;
  const int g = (lin / a.n_split_max) % nkv;
  const int row = lin / (a.n_split_max * nkv);
  const int Hq = a.num_q_heads;
  const int h0 = g * G;
  const int tid = threadIdx.x;

  int s, ctx;
  resolve_row(a, row, s, ctx);

  if (ctx <= 0) {   // no context: a zero row, written once
    if (split == 0) {
      for (int i = tid; i < G * kHeadDim; i += kThreads)
        store_out<BF16>(a.out, ((size_t)row * Hq + h0) * kHeadDim + i, 0.0f);
    }
    return;
  }
  const int nblk = (ctx + kBlockSize - 1) / kBlockSize;
  const int nsp = (nblk + SB - 1) / SB;
  if (split >= nsp) return;
  const int b_begin = split * SB;
  const int b_end = min(nblk, b_begin + SB);
  const int dirv = seq_direction(a.dir, a.cls, s);

  const int lane = tid & (kWave - 1);
  const int w = wave_id_uniform();
  const int R = lane >> 4;
  const int C = lane & 15;

  // This split's table entries, one per lane; read back wave-uniformly.
  int tbl = -1;
  if (b_begin + lane < b_end) tbl = a.block_tables[(size_t)s * a.max_blocks_per_seq + b_begin + lane];

  Frag<BF16> q[G];
#pragma unroll
  for (int h = 0; h < G; ++h) q[h].load(a.q, ((size_t)row * Hq + h0 + h) * kHeadDim + 8 * C);

  float m[G], l[G], acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = -INFINITY;
    l[h] = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = 0.0f;
  }

  const int nb_split = b_end - b_begin;
  const int nb_w = nb_split > w ? (nb_split - w + kWaves - 1) / kWaves : 0;
  const size_t lane_off = (size_t)R * kHeadDim + 8 * C;   // slot R, dims 8C.. (slot R+4j adds 4j rows)

  Frag<BF16> kc[4], vc[4];
  int blk_c = -1;
  auto load_tile = [&](int i, Frag<BF16>* kf, Frag<BF16>* vf) -> int {
    const int blk = read_lane_i32(tbl, w + kWaves * i);
    if (blk >= 0 && blk < a.num_blocks) {
      const size_t base = ((size_t)blk * nkv + g) * kTileElems + lane_off;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        kf[j].load(a.k_pool, base + (size_t)(4 * j) * kHeadDim);
        vf[j].load(a.v_pool, base + (size_t)(4 * j) * kHeadDim);
      }
      return blk;
    }
    return -1;
  };
  if (nb_w > 0) blk_c = load_tile(0, kc, vc);

  for (int i = 0; i < nb_w; ++i) {
    Frag<BF16> kn[4], vn[4];
    int blk_n = -1;
    if (i + 1 < nb_w) blk_n = load_tile(i + 1, kn, vn);

    if (blk_c >= 0) {
      const int b = b_begin + w + kWaves * i;       // logical block index
      float sc[G][4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
#pragma unroll
        for (int h = 0; h < G; ++h) sc[h][j] = row16_sum(q[h].dot(kc[j])) * a.scale_log2;
      }
      if (b == nblk - 1 && (ctx & (kBlockSize - 1)) != 0) {   // tail block: drop slots past the context
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int pos = b * kBlockSize + slot_of_offset(R + 4 * j, dirv);
          if (pos >= ctx) {
            vc[j].zero();
#pragma unroll
            for (int h = 0; h < G; ++h) sc[h][j] = -INFINITY;
          }
        }
      }
      float vv[4][8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
#pragma unroll
        for (int e = 0; e < 8; ++e) vv[j][e] = vc[j].at(e);
      }
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float mx = fmaxf(fmaxf(sc[h][0], sc[h][1]), fmaxf(sc[h][2], sc[h][3]));
        const float mnew = fmaxf(m[h], mx);
        const float mu = mnew == -INFINITY ? 0.0f : mnew;
        const float alpha = fast_exp2(m[h] - mu);
        const float p0 = fast_exp2(sc[h][0] - mu), p1 = fast_exp2(sc[h][1] - mu);
        const float p2 = fast_exp2(sc[h][2] - mu), p3 = fast_exp2(sc[h][3] - mu);
        l[h] = fmaf(l[h], alpha, (p0 + p1) + (p2 + p3));
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          float t = acc[h][e] * alpha;
          t = fmaf(p0, vv[0][e], t);
          t = fmaf(p1, vv[1][e], t);
          t = fmaf(p2, vv[2][e], t);
          acc[h][e] = fmaf(p3, vv[3][e], t);
        }
        m[h] = mnew;
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      kc[j] = kn[j];
      vc[j] = vn[j];
    }
    blk_c = blk_n;
  }

  // Merge the four 16-lane rows of the wave (lanes C, C+16, C+32, C+48 hold the
  // same head dims over disjoint slots).
#pragma unroll
  for (int xo = 16; xo <= 32; xo <<= 1) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float mo = __shfl_xor(m[h], xo);
      const float lo = __shfl_xor(l[h], xo);
      const float M = fmaxf(m[h], mo);
      const float mu = M == -INFINITY ? 0.0f : M;
      const float a1 = fast_exp2(m[h] - mu), a2 = fast_exp2(mo - mu);
      l[h] = l[h] * a1 + lo * a2;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] = acc[h][e] * a1 + __shfl_xor(acc[h][e], xo) * a2;
      m[h] = M;
    }
  }

  // Merge the four waves through LDS.
  __shared__ float s_acc[kWaves][G][kHeadDim];
  __shared__ float s_m[kWaves][G], s_l[kWaves][G];
  if (lane < 16) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
#pragma unroll
      for (int e = 0; e < 8; ++e) s_acc[w][h][8 * C + e] = acc[h][e];
    }
  }
  if (lane == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      s_m[w][h] = m[h];
      s_l[w][h] = l[h];
    }
  }
  __syncthreads();

  for (int idx = tid; idx < G * kHeadDim; idx += kThreads) {
    const int h = idx / kHeadDim;
    const int d = idx - h * kHeadDim;
    float M = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < kWaves; ++ww) M = fmaxf(M, s_m[ww][h]);
    const float mu = M == -INFINITY ? 0.0f : M;
    float L = 0.0f, A = 0.0f;
#pragma unroll
    for (int ww = 0; ww < kWaves; ++ww) {
      const float wt = fast_exp2(s_m[ww][h] - mu);
      L = fmaf(s_l[ww][h], wt, L);
      A = fmaf(s_acc[ww][h][d], wt, A);
    }
    const size_t qh = (size_t)row * Hq + h0 + h;
    if (nsp == 1) {
      store_out<BF16>(a.out, qh * kHeadDim + d, L > 0.0f ? A / L : 0.0f);
    } else {
      const size_t slot = qh * a.n_split_max + split;
      a.ws_acc[slot * kHeadDim + d] = A;
      if (d == 0) {
        a.ws_ml[2 * slot] = M;
        a.ws_ml[2 * slot + 1] = L;
      }
    }
  }
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
  float M = -INFINITY;
  for (int i = 0; i < nsp; ++i) M = fmaxf(M, a.ws_ml[2 * (base + i)]);
  const float mu = M == -INFINITY ? 0.0f : M;
  float L = 0.0f, A = 0.0f;
  for (int i = 0; i < nsp; ++i) {
    const float wt = fast_exp2(a.ws_ml[2 * (base + i)] - mu);
    L = fmaf(a.ws_ml[2 * (base + i) + 1], wt, L);
    A = fmaf(a.ws_acc[(base + i) * kHeadDim + d], wt, A);
  }
  store_out<BF16>(a.out, ((size_t)row * a.num_q_heads + hq) * kHeadDim + d, L > 0.0f ? A / L : 0.0f);
}

template <int G, bool BF16>
hipError_t launch_group(const DecodeArgs& a, hipStream_t stream) {
  const long long grid = (long long)a.num_rows * a.num_kv_heads * a.n_split_max;
  if (grid > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((decode_split_kernel<G, BF16>), dim3((unsigned)grid), dim3(kThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.n_split_max <= 1) return e;
  hipLaunchKernelGGL((decode_merge_kernel<BF16>), dim3((unsigned)(a.num_rows * a.num_q_heads)),
                     dim3(kHeadDim), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

DecodePlan plan_decode(int32_t num_rows, int32_t max_ctx) {
  DecodePlan p;
  const int64_t maxblk = max_ctx > 0 ? ((int64_t)max_ctx + kBlockSize - 1) / kBlockSize : 1;
  int sb = 32;   // 512 tokens per split by default
  while (sb > 4 && (int64_t)num_rows * ((maxblk + sb - 1) / sb) < 256) sb >>= 1;
  p.split_blocks = sb;
  p.n_split_max = (int32_t)((maxblk + sb - 1) / sb);
  return p;
}

size_t decode_workspace_bytes(int32_t num_rows, int32_t num_q_heads, int32_t max_ctx) {
  const DecodePlan p = plan_decode(num_rows, max_ctx);
  if (p.n_split_max <= 1) return 0;
  const size_t slots = (size_t)num_rows * num_q_heads * p.n_split_max;
  return slots * kHeadDim * sizeof(float) + slots * 2 * sizeof(float);
}

hipError_t launch_decode(DecodeArgs a, int group, bool bf16, hipStream_t stream) {
  switch (group * 2 + (bf16 ? 1 : 0)) {
    case 2: return launch_group<1, false>(a, stream);
    case 3: return launch_group<1, true>(a, stream);
    case 4: return launch_group<2, false>(a, stream);
    case 5: return launch_group<2, true>(a, stream);
    case 8: return launch_group<4, false>(a, stream);
    case 9: return launch_group<4, true>(a, stream);
    case 16: return launch_group<8, false>(a, stream);
    case 17: return launch_group<8, true>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace bros
