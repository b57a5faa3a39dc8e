// Lazy checkpointing on gfx950 (Sec. 5.2; the fetch/store kernels of Sec. 6):
// move the K/V rows of a list of slots between the pool and a dense buffer.
//
//   gather:  out[i][h][:] = pool[id_i / 16][h][id_i % 16][:]   (zero row when
//            id_i lies outside the pool)
//   scatter: pool[id_i / 16][h][id_i % 16][:] = in[i][h][:]     (skipped when
//            id_i lies outside the pool)
//
// for every KV head h, on both tensors. The dense side has the layout of a
// step's new tokens, [n][Hkv][D], so a checkpoint is one contiguous buffer
// that an asynchronous copy moves to or from pinned host memory while the
// compute units run attention. Pure byte movement in 16-byte chunks; each
// thread requests all of its chunks before it stores any.
#include "bros_device.h"
#include "bros_kernels.h"

namespace bros {
namespace {

constexpr int kThreads = 256;
constexpr int kIter = 8;   // 16-byte chunks per thread

typedef unsigned v4u_t __attribute__((ext_vector_type(4)));

template <bool GATHER>
__global__ __launch_bounds__(kThreads) void kv_move_kernel(KvMoveArgs a) {
  const int tid = threadIdx.x;
  const int64_t base = (int64_t)blockIdx.x * (kThreads * kIter);
  const int row_chunks = a.row_bytes / 16;                 // chunks of one (slot, head) row
  const int64_t per_tensor = (int64_t)a.num_kv_heads * row_chunks;
  const int64_t per_id = 2 * per_tensor;
  const int64_t total = (int64_t)a.num_slots * per_id;
  const int64_t pool_slots = (int64_t)a.num_blocks * kBlockSize;

  v4u_t data[kIter];
  int64_t dst[kIter];   // byte offset of the chunk's destination, -1 when skipped
  bool to_v[kIter];
#pragma unroll
  for (int it = 0; it < kIter; ++it) {
    const int64_t idx = base + (int64_t)it * kThreads + tid;
    dst[it] = -1;
    to_v[it] = false;
    if (idx >= total) continue;
    const int64_t i = idx / per_id;
    const int64_t rem = idx - i * per_id;
    const int tensor = rem >= per_tensor;                  // 0 = K, 1 = V
    const int64_t c = rem - tensor * per_tensor;           // chunk within the id's rows of that tensor
    const int64_t h = c / row_chunks;
    const int64_t cc = c - h * row_chunks;
    const int64_t sid = a.slot_ids[i];
    const bool inside = sid >= 0 && sid < pool_slots;
    const int64_t pool_off = (((sid / kBlockSize) * a.num_kv_heads + h) * kBlockSize + sid % kBlockSize) *
                                 (int64_t)a.row_bytes + cc * 16;
    const int64_t dense_off = (i * a.num_kv_heads + h) * (int64_t)a.row_bytes + cc * 16;
    to_v[it] = tensor != 0;
    if (GATHER) {
      const uint8_t* src = static_cast<const uint8_t*>(tensor ? a.v_pool : a.k_pool);
      data[it] = inside ? *reinterpret_cast<const v4u_t*>(src + pool_off) : v4u_t{0u, 0u, 0u, 0u};
      dst[it] = dense_off;
    } else if (inside) {
      const uint8_t* src = static_cast<const uint8_t*>(tensor ? a.v_dense : a.k_dense);
      data[it] = *reinterpret_cast<const v4u_t*>(src + dense_off);
      dst[it] = pool_off;
    }
  }
#pragma unroll
  for (int it = 0; it < kIter; ++it) {
    if (dst[it] < 0) continue;
    uint8_t* out = GATHER ? static_cast<uint8_t*>(to_v[it] ? a.v_dense : a.k_dense)
                          : static_cast<uint8_t*>(to_v[it] ? a.v_pool : a.k_pool);
    *reinterpret_cast<v4u_t*>(out + dst[it]) = data[it];
  }
}

}  // namespace

hipError_t launch_kv_move(const KvMoveArgs& a, bool gather, hipStream_t stream) {
  const int64_t total = (int64_t)a.num_slots * 2 * a.num_kv_heads * (a.row_bytes / 16);
  const int64_t grid = (total + kThreads * kIter - 1) / (kThreads * kIter);
  if (grid == 0) return hipSuccess;
  if (grid > 0x7fffffffLL) return hipErrorInvalidValue;
  if (gather)
    hipLaunchKernelGGL(kv_move_kernel<true>, dim3((unsigned)grid), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(kv_move_kernel<false>, dim3((unsigned)grid), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace bros
