// bros_kv_write on gfx950: store each new token's K/V rows in the slot its
// sequence's direction assigns (RT from the left end of a block, BE from the
// right end; Sec. 5.1), with the exclusive view of Sec. 5.2 (entry i of a
// sequence's table holds its positions [16 i, 16 i + 16)).
//
// One workgroup moves kTokens tokens. The first lanes resolve each token's
// destination (sequence by prefix search over cu_new staged in LDS, position,
// table entry, slot); then all 256 threads copy 16-byte chunks, every load of
// a thread issued before its first store. Writes are slot-granular, so two
// sequences sharing a block never race.
#include "bros_device.h"
#include "bros_kernels.h"

namespace bros {
namespace {

constexpr int kTokens = 8;          // tokens per workgroup
constexpr int kThreads = 256;
constexpr int kMaxSeqLds = 4096;    // prefix array staged in LDS up to this many sequences
constexpr int kMaxIter = 8;         // 16-byte chunks per thread per pass

template <bool BF16>
__global__ __launch_bounds__(kThreads) void kv_write_kernel(KvWriteArgs a) {
  __shared__ int s_cu[kMaxSeqLds + 1];
  __shared__ int s_dst[kTokens];   // block * 16 + slot, or -1 when the token is skipped

  const int tid = threadIdx.x;
  const int t0 = blockIdx.x * kTokens;
  const bool staged = a.num_seqs <= kMaxSeqLds;
  if (staged) {
    for (int i = tid; i <= a.num_seqs; i += kThreads) s_cu[i] = a.cu_new[i];
  }
  __syncthreads();

  if (tid < kTokens) {
    const int t = t0 + tid;
    int dst = -1;
    if (t < a.num_new_tokens) {
      int s = staged ? upper_index(s_cu, a.num_seqs + 1, t)
                     : upper_index(a.cu_new, a.num_seqs + 1, t);
      s = min(s, a.num_seqs - 1);   // a token past cu_new[num_seqs] stays in bounds
      const int first = staged ? s_cu[s] : a.cu_new[s];
      const int p = a.pos0[s] + (t - first);
      if (p >= 0) {
        const int bi = p >> 4;
        if (bi < a.max_blocks_per_seq) {
          const int blk = a.block_tables[(size_t)s * a.max_blocks_per_seq + bi];
          if (blk >= 0 && blk < a.num_blocks)
            dst = blk * kBlockSize + slot_of_offset(p & 15, seq_direction(a.dir, a.cls, s));
        }
      }
    }
    s_dst[tid] = dst;
  }
  __syncthreads();

  constexpr int kElem = BF16 ? 2 : 4;
  constexpr int kChunksPerRow = kHeadDim * kElem / 16;     // 16-byte chunks per head row
  const int chunks_per_token = a.num_kv_heads * kChunksPerRow;   // per tensor
  const int total = kTokens * 2 * chunks_per_token;
  const uint8_t* __restrict__ knew = static_cast<const uint8_t*>(a.k_new);
  const uint8_t* __restrict__ vnew = static_cast<const uint8_t*>(a.v_new);
  uint8_t* __restrict__ kpool = static_cast<uint8_t*>(a.k_pool);
  uint8_t* __restrict__ vpool = static_cast<uint8_t*>(a.v_pool);
  const size_t row_bytes = (size_t)kHeadDim * kElem;

  for (int base = 0; base < total; base += kThreads * kMaxIter) {
    uint4 data[kMaxIter];
    size_t dst_off[kMaxIter];
    bool live[kMaxIter];
    bool is_v[kMaxIter];
#pragma unroll
    for (int it = 0; it < kMaxIter; ++it) {
      const int idx = base + it * kThreads + tid;
      live[it] = false;
      is_v[it] = false;
      dst_off[it] = 0;
      if (idx < total) {
        const int tok = idx / (2 * chunks_per_token);
        const int rem = idx - tok * 2 * chunks_per_token;
        const int tensor = rem / chunks_per_token;          // 0 = K, 1 = V
        const int c = rem - tensor * chunks_per_token;
        const int h = c / kChunksPerRow;
        const int cc = c - h * kChunksPerRow;
        const int dst = s_dst[tok];
        if (dst >= 0 && t0 + tok < a.num_new_tokens) {
          const size_t src_off = ((size_t)(t0 + tok) * a.num_kv_heads + h) * row_bytes + (size_t)cc * 16;
          data[it] = *reinterpret_cast<const uint4*>((tensor ? vnew : knew) + src_off);
          const int blk = dst >> 4, slot = dst & 15;
          dst_off[it] = (((size_t)blk * a.num_kv_heads + h) * kBlockSize + slot) * row_bytes + (size_t)cc * 16;
          live[it] = true;
          is_v[it] = tensor != 0;
        }
      }
    }
#pragma unroll
    for (int it = 0; it < kMaxIter; ++it) {
      if (live[it]) *reinterpret_cast<uint4*>((is_v[it] ? vpool : kpool) + dst_off[it]) = data[it];
    }
  }
}

}  // namespace

hipError_t launch_kv_write(const KvWriteArgs& a, bool bf16, hipStream_t stream) {
  const int grid = (a.num_new_tokens + kTokens - 1) / kTokens;
  if (grid == 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(kv_write_kernel<true>, dim3(grid), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(kv_write_kernel<false>, dim3(grid), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace bros
