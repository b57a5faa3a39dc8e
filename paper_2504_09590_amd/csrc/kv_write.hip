// bros_kv_write on gfx950: store each new token's K/V rows in the slot its
// block's direction assigns (RT from the left end of a block, BE from the
// right end; Sec. 5.1), with the exclusive view of Sec. 5.2 (entry i of a
// sequence's table holds its positions [16 i, 16 i + 16)). The direction is
// the sequence's, or that of the token's table entry (Sec. 6's table).
//
// One workgroup moves kTokens tokens. Its 256 threads first request their
// sequence ranges and the tokens' source rows (16-byte chunks), which do not
// depend on the destination; each thread then checks one sequence's range of
// new tokens, and one thread per token resolves its destination (position,
// table entry, slot); then the chunks are stored. Writes are
// slot-granular, so two sequences sharing a block never race.
#include "bros_device.h"
#include "bros_kernels.h"

namespace bros {
namespace {

// Tokens per workgroup, and 16-byte chunks per thread per pass (Hkv 8, bf16:
// one pass). Two tokens, two chunks per thread measured fastest (kernel 5.0
// us for 2176 tokens against 5.6 us with four tokens, four chunks per thread;
// one chunk per thread, or 8 to 16 tokens per workgroup, were slower).
constexpr int kTokens = 2;
constexpr int kThreads = 256;
constexpr int kMaxIter = 2;

typedef unsigned v4u_t __attribute__((ext_vector_type(4)));   // 16 bytes (a plain vector promotes to registers)

// n / d for 0 <= n < 2^22 and d >= 1, with rcp = 1 / d: the float estimate is
// within one of the quotient, and one correction step makes it exact (a few
// instructions instead of the long integer division sequence).
__device__ __forceinline__ int div_small(int n, int d, float rcp) {
  int q = (int)((float)n * rcp);
  const int r = n - q * d;
  q += (r >= d) ? 1 : 0;
  q -= (r < 0) ? 1 : 0;
  return q;
}

template <bool BF16>
__global__ __launch_bounds__(kThreads) void kv_write_kernel(KvWriteArgs a) {
  __shared__ int s_seq[kTokens];   // the sequence holding each token, or -1
  __shared__ int s_pos[kTokens];   // the token's position in it
  __shared__ int s_dst[kTokens];   // block * 16 + slot, or -1 when the token is skipped

  const int tid = threadIdx.x;
  const int t0 = blockIdx.x * kTokens;

  constexpr int kElem = BF16 ? 2 : 4;
  constexpr int kChunksPerRow = kHeadDim * kElem / 16;     // 16-byte chunks per head row
  const int chunks_per_token = a.num_kv_heads * kChunksPerRow;   // per tensor
  const int total = kTokens * 2 * chunks_per_token;
  const float rcp_cpt = 1.0f / (float)chunks_per_token;
  const uint8_t* __restrict__ knew = static_cast<const uint8_t*>(a.k_new);
  const uint8_t* __restrict__ vnew = static_cast<const uint8_t*>(a.v_new);
  uint8_t* __restrict__ kpool = static_cast<uint8_t*>(a.k_pool);
  uint8_t* __restrict__ vpool = static_cast<uint8_t*>(a.v_pool);
  constexpr uint32_t kRowBytes = kHeadDim * kElem;
  const int n_tok = min(kTokens, a.num_new_tokens - t0);   // tokens of this workgroup (>= 1)

  // Chunk idx of the workgroup: (token, tensor) pair tt = idx / chunks_per_token
  // (token tt / 2, tensor tt % 2: 0 = K, 1 = V), chunk c within the token's
  // rows. `part` is its offset inside a block's rows for that KV head:
  // (h * 16 slots) rows plus the chunk within the row.
  struct Chunk {
    int tok, tensor, c;
    uint32_t part;
    bool live;
  };
  auto split = [&](int idx) -> Chunk {
    Chunk k;
    const int tt = div_small(idx, chunks_per_token, rcp_cpt);
    k.c = idx - tt * chunks_per_token;
    k.tok = tt >> 1;
    k.tensor = tt & 1;
    const int h = k.c / kChunksPerRow, cc = k.c % kChunksPerRow;   // (constant divisor: a shift)
    k.part = ((uint32_t)h * kBlockSize) * kRowBytes + (uint32_t)cc * 16;
    k.live = idx < total && k.tok < n_tok;
    return k;
  };

  // This thread's first sequence range (thread j: sequence j), requested
  // before the source rows: loads return in order, so the range check below
  // then waits for these alone, not for the rows coming from HBM.
  int m_lo = 0, m_hi = 0, m_p0 = 0;
  if (tid < a.num_seqs) {
    m_lo = a.cu_new[tid];
    m_hi = a.cu_new[tid + 1];
    m_p0 = a.pos0[tid];
  }
  // Source rows of the first pass: they do not depend on where the tokens go,
  // so they are requested before the destinations are resolved.
  v4u_t data[kMaxIter];
  Chunk ch[kMaxIter];
#pragma unroll
  for (int it = 0; it < kMaxIter; ++it) {
    ch[it] = split(it * kThreads + tid);
    if (ch[it].live)
      data[it] = *reinterpret_cast<const v4u_t*>((ch[it].tensor ? vnew : knew) +
                                                   ((size_t)(t0 + ch[it].tok) * chunks_per_token + ch[it].c) * 16);
  }

  // Destinations, in two rounds of loads. First, thread j checks whether
  // sequence j holds any of this workgroup's tokens (its prefix offsets and
  // first position) and notes, per token it holds, the sequence and position.
  // Then thread t < kTokens resolves token t's table entry and direction, so
  // that the tokens' lookups run side by side. A token in no sequence's
  // range is skipped.
  if (tid < kTokens) s_seq[tid] = -1;
  __syncthreads();
  for (int j = tid; j < a.num_seqs; j += kThreads) {
    const bool first = j == tid;
    const int lo = first ? m_lo : a.cu_new[j], hi = first ? m_hi : a.cu_new[j + 1];
    const int p0 = first ? m_p0 : a.pos0[j];
    const int k0 = max(lo, t0), k1 = min(hi, t0 + n_tok);
    for (int k = k0; k < k1; ++k) {
      s_seq[k - t0] = j;
      s_pos[k - t0] = p0 + (k - lo);
    }
  }
  __syncthreads();
  if (tid < kTokens) {
    const int j = s_seq[tid], p = s_pos[tid];
    int dst = -1;
    if (j >= 0 && p >= 0 && (p >> 4) < a.max_blocks_per_seq) {
      const int blk = a.block_tables[(size_t)j * a.max_blocks_per_seq + (p >> 4)];
      const int dirv = entry_direction(a.dir, a.cls, a.dir_per_entry, a.max_blocks_per_seq, j, p >> 4);
      if (blk >= 0 && blk < a.num_blocks) dst = blk * kBlockSize + slot_of_offset(p & 15, dirv);
    }
    s_dst[tid] = dst;
  }
  __syncthreads();

  // Store one pass's chunks to their slots: row (blk * Hkv + h) * 16 + slot.
  auto store = [&](const Chunk& k, const v4u_t& v) {
    if (!k.live) return;
    const int dst = s_dst[k.tok];
    if (dst < 0) return;
    const size_t row0 = (size_t)(dst >> 4) * a.num_kv_heads * kBlockSize + (dst & 15);   // h = 0
    *reinterpret_cast<v4u_t*>((k.tensor ? vpool : kpool) + row0 * kRowBytes + k.part) = v;
  };
#pragma unroll
  for (int it = 0; it < kMaxIter; ++it) store(ch[it], data[it]);
  // Further passes (more KV heads than one pass holds): load, then store.
  for (int base = kThreads * kMaxIter; base < total; base += kThreads * kMaxIter) {
    v4u_t more[kMaxIter];
    Chunk mk[kMaxIter];
#pragma unroll
    for (int it = 0; it < kMaxIter; ++it) {
      mk[it] = split(base + it * kThreads + tid);
      if (mk[it].live)
        more[it] = *reinterpret_cast<const v4u_t*>((mk[it].tensor ? vnew : knew) +
                                                     ((size_t)(t0 + mk[it].tok) * chunks_per_token + mk[it].c) * 16);
    }
#pragma unroll
    for (int it = 0; it < kMaxIter; ++it) store(mk[it], more[it]);
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
