// Pieces shared by the two decode paths: bf16 on the matrix cores
// (decode.hip) and fp32 on the vector ALU (decode_f32.hip).
#pragma once

#include "bros_device.h"
#include "bros_kernels.h"

#include <math.h>

namespace bros {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kTileElems = kBlockSize * kHeadDim;   // one (block, KV head) tile
constexpr float kRescaleSlack = 8.0f;               // log2 units: weights stay <= 2^8
constexpr float kNoMax = -1.0e30f;                  // finite "no score yet" reference
constexpr int kMaxRowsLds = 4096;                   // rows whose prefix fits in LDS

typedef unsigned v4u_t __attribute__((ext_vector_type(4)));

// Lane id through an asm the compiler cannot hoist: values derived from it are
// recomputed where they are used instead of being held in registers.
__device__ __forceinline__ int lane_id_here() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {   // round to nearest even
  typedef __attribute__((__vector_size__(2 * sizeof(float)))) float f2_t;
  typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 b2_t;
  const f2_t f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, b2_t));
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

hipError_t launch_decode_f32(const DecodeArgs& a, int group, hipStream_t stream);

}  // namespace bros
