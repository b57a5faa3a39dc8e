// bros_attn_decode_noalloc: bros_attn_decode with its workspace in a static
// device array, for callers that cannot allocate device memory (code under
// HIP graph capture, serving loops and harnesses that forbid hipMalloc).
//
// The array is a file-scope __device__ object: every GPU the library runs on
// holds its own copy, at its own address, from the code object's load until
// the process ends. Host code never passes the array's name to a kernel (in
// host code that name is only a stand-in for the symbol); the first call on a
// device resolves that device's address with hipGetSymbolAddress, with the
// device current, and every later call on the device uses the stored address.
// Calls on one GPU share its array: two calls that overlap in time on one GPU
// race on it. Nothing in it has to start at zero (the decode kernel writes
// every partial and row prefix before its merge reads them).
#include "bros_attn.h"
#include "bros_error.h"
#include "bros_kernels.h"

#include <hip/hip_runtime.h>

#include <mutex>

namespace {

__device__ __align__(256) unsigned char scratch[BROS_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
void* g_scratch[kMaxDevices];   // per device: the address of that device's copy of `scratch`
std::mutex g_scratch_mu;

// Address of the current device's copy of `scratch` (resolved once per device).
int scratch_address(const char* fn, void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return bros::fail(BROS_E_HIP, "%s: hipGetDevice: %s", fn, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return bros::fail(BROS_E_UNSUPPORTED, "%s: device %d beyond the %d supported", fn, dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return bros::fail(BROS_E_HIP, "%s: hipGetSymbolAddress of the scratch array on device %d: %s", fn, dev,
                        e != hipSuccess ? hipGetErrorString(e) : "null address");
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return BROS_OK;
}

}  // namespace

extern "C" int bros_attn_decode_noalloc(void* out, const void* q,
                                        const void* k_pool, const void* v_pool, int32_t num_blocks,
                                        const int32_t* block_tables, int32_t max_blocks_per_seq,
                                        const int8_t* dir, const uint8_t* cls, int32_t dir_per_entry,
                                        const int32_t* ctx_lens, int32_t max_ctx, int32_t num_seqs,
                                        int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                        int32_t block_size, float scale, int32_t dtype, void* stream) {
  const char* fn = "bros_attn_decode_noalloc";
  // The size query returns 0 for unsupported arguments; bros_attn_decode then
  // reports them without launching anything.
  const size_t need = bros_attn_workspace_size(BROS_WS_DECODE, dtype, num_seqs, num_q_heads, head_dim, max_ctx);
  if (need > (size_t)BROS_NOALLOC_SCRATCH_BYTES)
    return bros::fail(BROS_E_WORKSPACE,
                      "%s: this batch needs %zu bytes of workspace; the static scratch array holds %zu "
                      "(use bros_attn_decode with a workspace of that size)",
                      fn, need, (size_t)BROS_NOALLOC_SCRATCH_BYTES);
  // A call with a missing tensor is reported by bros_attn_decode's own checks
  // before any HIP call; only a call that can launch resolves the array.
  const bool launchable = out && q && k_pool && v_pool && ctx_lens && block_tables && (dir || cls);
  void* ws = nullptr;
  if (need > 0 && num_seqs > 0 && launchable) {
    const int st = scratch_address(fn, &ws);
    if (st != BROS_OK) return st;
  }
  return bros_attn_decode(out, q, k_pool, v_pool, num_blocks, block_tables, max_blocks_per_seq, dir, cls,
                          dir_per_entry, ctx_lens, max_ctx, num_seqs, num_q_heads, num_kv_heads, head_dim,
                          block_size, scale, dtype, ws, ws != nullptr ? (size_t)BROS_NOALLOC_SCRATCH_BYTES : 0,
                          stream);
}
