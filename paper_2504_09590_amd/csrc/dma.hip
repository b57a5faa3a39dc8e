// Host copies on a copy (SDMA) engine, ordered against a HIP stream.
//
// Whether hipMemcpyAsync runs on a copy engine or as a copy kernel is the HIP
// runtime's choice, and the runtime bundled with PyTorch for ROCm 7.0 makes a
// kernel of every copy, which then takes compute units from the attention or
// queues behind it. Here the copy goes straight to a copy engine through the
// ROCr runtime that the HIP runtime itself has loaded
// (hsa_amd_memory_async_copy_on_engine), and two HSA signals order it against
// the stream:
//   start  the engine begins the copy once it reads 0; a one-lane kernel on
//          the stream stores the 0 when the stream's earlier work is done;
//   done   the engine decrements it from 1 to 0 when the copy has landed; a
//          one-lane kernel on the stream waits for the 0 before the stream's
//          later work, sleeping between polls so that it takes next to no
//          issue slots from the kernels beside it, then stores 2 into start.
// That 2 tells the host the pair is free: a pair is re-armed (both set to 1)
// only after the host has read it, so a stream never waits on a pair that a
// later copy re-armed. Pairs live in a pool that grows to the number of
// copies in flight; nothing on the host waits for the device.
//
// Progress: a copy waits in its engine's queue behind the copies requested
// before it, and each of those waits only for stream work enqueued before it
// was requested; every wait therefore ends. The wait kernel still gives up
// after kWaitLimitTicks (it then raises a flag that the next call reports).
// HIP's own stream memory operations would serve too, but the ROCm 7.0
// runtime implements the wait as a kernel that polls without sleeping.
#include "bros_attn.h"
#include "bros_error.h"

#include <hip/hip_runtime.h>
#include <hsa/amd_hsa_signal.h>
#include <hsa/hsa.h>
#include <hsa/hsa_ext_amd.h>

#include <dlfcn.h>
#include <cinttypes>
#include <link.h>

#include <algorithm>
#include <chrono>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

namespace {

using bros::fail;
using bros::ok;

struct Rocr {
  hsa_status_t (*iterate_agents)(hsa_status_t (*)(hsa_agent_t, void*), void*);
  hsa_status_t (*agent_get_info)(hsa_agent_t, hsa_agent_info_t, void*);
  hsa_status_t (*engine_status)(hsa_agent_t, hsa_agent_t, uint32_t*);
  hsa_status_t (*signal_create)(hsa_signal_value_t, uint32_t, const hsa_agent_t*, hsa_signal_t*);
  hsa_signal_value_t (*signal_load)(hsa_signal_t);
  void (*signal_store)(hsa_signal_t, hsa_signal_value_t);
  hsa_status_t (*copy_on_engine)(void*, hsa_agent_t, const void*, hsa_agent_t, size_t, uint32_t, const hsa_signal_t*,
                                 hsa_signal_t, hsa_amd_sdma_engine_id_t, bool);
};

struct GpuAgent {
  uint32_t domain = 0, bdf = 0;
  hsa_agent_t agent{0};
};

struct GpuEngines {
  hsa_agent_t gpu{0};
  uint32_t h2d = 1, d2h = 2, d2d = 4;
};

struct State {
  std::mutex mu;
  std::vector<GpuEngines> engines;
  bool tried = false;
  std::string error;            // why the engines cannot be used ("" once ready)
  Rocr r{};
  hsa_agent_t cpu{0};
  std::vector<GpuAgent> gpus;
  struct Pair {
    hsa_signal_t start, done;
    bool issued;   // a copy was handed to an engine with this pair
    bool dead;     // its copy never ended: never reused
  };
  std::vector<Pair> pairs;
  size_t next = 0;
  int32_t* timed_out = nullptr;   // pinned host word the wait kernel raises
};

State& state() {
  static State s;
  return s;
}

// Every loaded ROCr library (normally one: the HIP runtime's).
int collect_rocr(struct dl_phdr_info* info, size_t, void* out) {
  if (info->dlpi_name && std::strstr(info->dlpi_name, "libhsa-runtime64"))
    static_cast<std::vector<std::string>*>(out)->push_back(info->dlpi_name);
  return 0;
}

std::string dir_of(const std::string& p) { return p.substr(0, p.find_last_of('/') + 1); }

hsa_status_t collect_agent(hsa_agent_t a, void* arg) {
  State& s = *static_cast<State*>(arg);
  hsa_device_type_t t;
  if (s.r.agent_get_info(a, HSA_AGENT_INFO_DEVICE, &t) != HSA_STATUS_SUCCESS) return HSA_STATUS_SUCCESS;
  if (t == HSA_DEVICE_TYPE_CPU && s.cpu.handle == 0) s.cpu = a;
  if (t == HSA_DEVICE_TYPE_GPU) {
    GpuAgent g;
    g.agent = a;
    s.r.agent_get_info(a, (hsa_agent_info_t)HSA_AMD_AGENT_INFO_DOMAIN, &g.domain);
    s.r.agent_get_info(a, (hsa_agent_info_t)HSA_AMD_AGENT_INFO_BDFID, &g.bdf);
    s.gpus.push_back(g);
  }
  return HSA_STATUS_SUCCESS;
}

// Binds to the ROCr instance the HIP runtime uses: the one in the HIP
// library's directory if several are loaded, else the first that has agents.
void bind_rocr(State& s) {
  s.tried = true;
  std::vector<std::string> libs;
  dl_iterate_phdr(collect_rocr, &libs);
  Dl_info hip{};
  const std::string hip_dir = dladdr(reinterpret_cast<void*>(&hipStreamWriteValue64), &hip) && hip.dli_fname
                                  ? dir_of(hip.dli_fname) : std::string();
  std::stable_partition(libs.begin(), libs.end(), [&](const std::string& p) { return dir_of(p) == hip_dir; });
  for (const std::string& path : libs) {
    void* h = dlopen(path.c_str(), RTLD_NOW | RTLD_NOLOAD);
    if (h == nullptr) continue;
    Rocr r{};
    r.iterate_agents = reinterpret_cast<decltype(r.iterate_agents)>(dlsym(h, "hsa_iterate_agents"));
    r.agent_get_info = reinterpret_cast<decltype(r.agent_get_info)>(dlsym(h, "hsa_agent_get_info"));
    r.engine_status = reinterpret_cast<decltype(r.engine_status)>(dlsym(h, "hsa_amd_memory_copy_engine_status"));
    r.signal_create = reinterpret_cast<decltype(r.signal_create)>(dlsym(h, "hsa_signal_create"));
    r.signal_load = reinterpret_cast<decltype(r.signal_load)>(dlsym(h, "hsa_signal_load_scacquire"));
    r.signal_store = reinterpret_cast<decltype(r.signal_store)>(dlsym(h, "hsa_signal_store_screlease"));
    r.copy_on_engine = reinterpret_cast<decltype(r.copy_on_engine)>(dlsym(h, "hsa_amd_memory_async_copy_on_engine"));
    dlclose(h);   // RTLD_NOLOAD took a reference of a library that stays loaded
    if (!r.iterate_agents || !r.agent_get_info || !r.engine_status || !r.signal_create || !r.signal_load ||
        !r.signal_store || !r.copy_on_engine)
      continue;
    s.r = r;
    s.cpu = hsa_agent_t{0};
    s.gpus.clear();
    if (r.iterate_agents(collect_agent, &s) == HSA_STATUS_SUCCESS && s.cpu.handle != 0 && !s.gpus.empty()) {
      void* word = nullptr;
      if (hipHostMalloc(&word, 64, hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess || word == nullptr) {
        s.error = "hipHostMalloc of the wait flag failed";
        return;
      }
      s.timed_out = static_cast<int32_t*>(word);
      *s.timed_out = 0;
      s.error.clear();
      return;
    }
  }
  s.error = libs.empty() ? "no ROCr library is loaded" : "no loaded ROCr library has a CPU and a GPU agent";
}

// The ROCr agent of HIP device `dev`, found by its PCI location.
bool gpu_agent(State& s, int dev, hsa_agent_t* out) {
  int bus = 0, slot = 0, domain = 0;
  if (hipDeviceGetAttribute(&bus, hipDeviceAttributePciBusId, dev) != hipSuccess ||
      hipDeviceGetAttribute(&slot, hipDeviceAttributePciDeviceId, dev) != hipSuccess ||
      hipDeviceGetAttribute(&domain, hipDeviceAttributePciDomainID, dev) != hipSuccess)
    return false;
  for (const GpuAgent& g : s.gpus)
    if (g.domain == (uint32_t)domain && (g.bdf >> 8) == (uint32_t)bus && ((g.bdf >> 3) & 31u) == (uint32_t)slot) {
      *out = g.agent;
      return true;
    }
  if (s.gpus.size() == 1) {   // one GPU: no choice to make
    *out = s.gpus[0].agent;
    return true;
  }
  return false;
}

// The agent that owns `p`: its device's GPU agent, or the CPU agent for
// pinned host memory. Pageable host memory is refused.
int owner(State& s, const char* fn, const char* what, const void* p, hsa_agent_t* agent, bool* is_host) {
  hipPointerAttribute_t a{};
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return fail(BROS_E_SHAPE, "%s: %s is neither device memory nor pinned host memory", fn, what);
  }
  if (a.type == hipMemoryTypeHost) {
    *agent = s.cpu;
    *is_host = true;
    return BROS_OK;
  }
  if (a.type == hipMemoryTypeDevice || a.type == hipMemoryTypeManaged) {
    *is_host = false;
    if (!gpu_agent(s, a.device, agent)) return fail(BROS_E_HIP, "%s: no ROCr agent for device %d", fn, a.device);
    return BROS_OK;
  }
  return fail(BROS_E_SHAPE, "%s: %s is neither device memory nor pinned host memory", fn, what);
}

// Engines per GPU, chosen once while they are idle and then kept: host-to-
// device on the first engine the pair reports, device-to-host on the next,
// device-to-device on the one after. The availability mask changes while
// copies are in flight, and moving an engine from one direction to another
// makes the runtime wait for it on the host.
uint32_t lowest_bit(uint32_t m) { return m & (~m + 1u); }

uint32_t pick_engine(State& s, hsa_agent_t gpu, bool to_host, bool from_host) {
  for (const GpuEngines& g : s.engines)
    if (g.gpu.handle == gpu.handle) return from_host ? g.h2d : to_host ? g.d2h : g.d2d;
  uint32_t h2d_mask = 0, d2h_mask = 0;
  if (s.r.engine_status(gpu, s.cpu, &h2d_mask) != HSA_STATUS_SUCCESS || h2d_mask == 0) h2d_mask = 0x7u;
  if (s.r.engine_status(s.cpu, gpu, &d2h_mask) != HSA_STATUS_SUCCESS || d2h_mask == 0) d2h_mask = 0x7u;
  GpuEngines g;
  g.gpu = gpu;
  g.h2d = lowest_bit(h2d_mask);
  g.d2h = lowest_bit(d2h_mask & ~g.h2d) ? lowest_bit(d2h_mask & ~g.h2d) : lowest_bit(d2h_mask);
  const uint32_t rest = (h2d_mask | d2h_mask) & ~(g.h2d | g.d2h);
  g.d2d = rest ? lowest_bit(rest) : g.h2d;
  s.engines.push_back(g);
  return from_host ? g.h2d : to_host ? g.d2h : g.d2d;
}

constexpr int64_t kArmed = 1, kGo = 0, kFree = 2;
constexpr uint64_t kWaitLimitTicks = 100ull * 1000 * 1000 * 10;   // 10 s of the 100 MHz real-time counter
constexpr double kLinkPeakBytesPerTick = 64e9 / 100e6;              // no copy is faster than 64 GB/s

__global__ void dma_go_kernel(int64_t* start) {
  if (threadIdx.x == 0) __hip_atomic_store(start, kGo, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Polls of pinned host memory are not free for the kernels beside the wait:
// one wave polling every half microsecond slows an HBM-bound grid on the
// other compute units by about a fifth (measured on MI355X). So the wait
// first sleeps, without a poll, for the shortest time the copy can take
// (quiet_ticks, from its size at the host link's peak), and then polls only
// every few microseconds.
__global__ void dma_wait_kernel(const int64_t* done, int64_t* start, int32_t* timed_out, uint64_t quiet_ticks) {
  if (threadIdx.x != 0) return;
  const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
  while (__builtin_amdgcn_s_memrealtime() - t0 < quiet_ticks) __builtin_amdgcn_s_sleep(127);
  // relaxed polls (an acquire would invalidate the cache on every poll),
  // one acquire fence once the copy has landed
  while (__hip_atomic_load(done, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) != 0) {
    if (__builtin_amdgcn_s_memrealtime() - t0 > kWaitLimitTicks) {
      __hip_atomic_store(timed_out, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      return;
    }
    __builtin_amdgcn_s_sleep(127);   // about 3.4 us at 2.4 GHz
  }
  __atomic_thread_fence(__ATOMIC_ACQUIRE);
  __hip_atomic_store(start, kFree, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

int64_t* value_of(hsa_signal_t sig) { return const_cast<int64_t*>(&reinterpret_cast<amd_signal_t*>(sig.handle)->value); }

}  // namespace

extern "C" int bros_copy_dma(void* dst, const void* src, size_t bytes, void* stream) {
  const char* fn = "bros_copy_dma";
  if (bytes == 0) return ok();
  if (dst == nullptr || src == nullptr) return fail(BROS_E_NULL, "%s: dst or src is NULL", fn);
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(static_cast<hipStream_t>(stream), &cap) != hipSuccess) (void)hipGetLastError();
  if (cap != hipStreamCaptureStatusNone)
    return fail(BROS_E_UNSUPPORTED, "%s: the stream is being captured; an engine copy is not part of a graph", fn);
  State& s = state();
  std::lock_guard<std::mutex> lock(s.mu);
  if (!s.tried) bind_rocr(s);
  if (!s.error.empty()) return fail(BROS_E_HIP, "%s: copy engines unavailable: %s", fn, s.error.c_str());
  if (__atomic_load_n(s.timed_out, __ATOMIC_ACQUIRE) != 0)
    return fail(BROS_E_HIP, "%s: an earlier copy did not end within the wait limit; its stream went on unordered", fn);
  hsa_agent_t da{0}, sa{0};
  bool dst_host = false, src_host = false;
  int st = owner(s, fn, "dst", dst, &da, &dst_host);
  if (st == BROS_OK) st = owner(s, fn, "src", src, &sa, &src_host);
  if (st != BROS_OK) return st;
  if (dst_host && src_host) return fail(BROS_E_SHAPE, "%s: host-to-host copy (one side must be device memory)", fn);
  const uint32_t engine = pick_engine(s, dst_host ? sa : da, dst_host, src_host);

  // a free pair: one whose stream has written kFree, or a new one
  State::Pair* p = nullptr;
  for (size_t i = 0; i < s.pairs.size() && p == nullptr; ++i) {
    State::Pair& c = s.pairs[(s.next + i) % s.pairs.size()];
    if (!c.dead && (!c.issued || s.r.signal_load(c.start) == kFree)) {
      p = &c;
      s.next = (s.next + i + 1) % s.pairs.size();
    }
  }
  if (p == nullptr) {
    State::Pair c{};
    if (s.r.signal_create(kArmed, 0, nullptr, &c.start) != HSA_STATUS_SUCCESS ||
        s.r.signal_create(kArmed, 0, nullptr, &c.done) != HSA_STATUS_SUCCESS)
      return fail(BROS_E_HIP, "%s: hsa_signal_create failed", fn);
    s.pairs.push_back(c);
    p = &s.pairs.back();
  }
  s.r.signal_store(p->done, kArmed);
  s.r.signal_store(p->start, kArmed);
  const hsa_status_t hs = s.r.copy_on_engine(dst, da, src, sa, bytes, 1, &p->start, p->done,
                                             static_cast<hsa_amd_sdma_engine_id_t>(engine), true);
  if (hs != HSA_STATUS_SUCCESS) {
    p->issued = false;
    return fail(BROS_E_HIP, "%s: hsa_amd_memory_async_copy_on_engine of %zu bytes failed (status 0x%x)", fn, bytes,
                (unsigned)hs);
  }
  p->issued = true;
  hipStream_t hst = static_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(dma_go_kernel, dim3(1), dim3(64), 0, hst, value_of(p->start));
  hipError_t e = hipGetLastError();
  if (e == hipSuccess) {
    const uint64_t quiet = (dst_host || src_host) ? (uint64_t)((double)bytes / kLinkPeakBytesPerTick) : 0;
    hipLaunchKernelGGL(dma_wait_kernel, dim3(1), dim3(64), 0, hst, value_of(p->done), value_of(p->start),
                       s.timed_out, quiet);
    e = hipGetLastError();
  }
  if (e != hipSuccess) {
    // The copy is queued on the engine but the stream cannot order it: let it
    // run after the stream's current work, and wait for it here.
    const char* why = hipGetErrorString(e);
    (void)hipStreamSynchronize(hst);
    s.r.signal_store(p->start, kGo);
    const auto t0 = std::chrono::steady_clock::now();
    while (s.r.signal_load(p->done) != 0) {
      if (std::chrono::steady_clock::now() - t0 > std::chrono::seconds(10)) {
        p->dead = true;   // the engine may still hold it
        return fail(BROS_E_HIP, "%s: ordering the copy on the stream failed (%s) and the copy did not end", fn, why);
      }
    }
    s.r.signal_store(p->start, kFree);
    return fail(BROS_E_HIP, "%s: ordering the copy on the stream failed (%s); it was completed synchronously", fn, why);
  }
  return ok();
}
