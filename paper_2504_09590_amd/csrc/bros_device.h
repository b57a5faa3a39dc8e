// Device helpers shared by the gfx950 kernels of the bidirectional paged-attention step.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bros {

constexpr int kBlockSize = 16;   // slots per KV block
constexpr int kHeadDim = 128;    // supported head dimension
constexpr int kWave = 64;        // CDNA wavefront width

// Slot of in-block offset `off` for a sequence walking its blocks in direction
// `dir` (+1 from the left end, -1 from the right end); its own inverse.
__device__ __forceinline__ int slot_of_offset(int off, int dir) {
  return dir > 0 ? off : (kBlockSize - 1 - off);
}

// Direction of sequence s: the explicit flag when given, else from the class
// (RT fills from the left, BE from the right).
__device__ __forceinline__ int seq_direction(const int8_t* dir, const uint8_t* cls, int s) {
  if (dir != nullptr) return dir[s] < 0 ? -1 : 1;
  return cls[s] == 1 ? -1 : 1;
}

// Direction of block-table entry e of sequence s. With per_entry set, dir is
// the paper's direction table, shaped like the block tables ([S][max_blocks],
// Sec. 6); otherwise one flag per sequence (or the class when dir is NULL).
__device__ __forceinline__ int entry_direction(const int8_t* dir, const uint8_t* cls, int per_entry,
                                               int max_blocks, int s, int e) {
  if (dir != nullptr && per_entry) return dir[(size_t)s * max_blocks + e] < 0 ? -1 : 1;
  return seq_direction(dir, cls, s);
}

// bf16 <-> fp32. Widening is exact (a shift); narrowing rounds to nearest-even
// and keeps NaNs quiet.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;  // NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return f32_to_bf16_bits(lo) | (f32_to_bf16_bits(hi) << 16);
}

// Base-2 exponential on the transcendental unit (exp2(-inf) = 0).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ int wave_id_uniform() {
  return __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
}

__device__ __forceinline__ int read_lane_i32(int v, int lane) {
  return __builtin_amdgcn_readlane(v, lane);
}

// Largest i in [0, n) with a[i] <= key, for a non-decreasing device array
// (finds the sequence a flattened row belongs to from prefix offsets).
__device__ __forceinline__ int upper_index(const int32_t* a, int n, int key) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (a[mid] <= key) lo = mid; else hi = mid - 1;
  }
  return lo;
}

}  // namespace bros
