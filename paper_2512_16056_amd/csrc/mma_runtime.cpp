// Host side of the multipath copy path on ROCr/HIP: the C ABI (the paper's
// Transfer Task Interceptor, Section 3.2: record the request, plan it, enqueue
// the dummy task on the stream), argument validation against the HIP pointer
// attributes, the engine backend that issues SDMA commands through ROCr, and
// the kernel launches. The engine itself (path selection, completion
// accounting, the CU-ring protocol) is in mma_engine.h.
#include <hip/hip_runtime.h>
#include <hsa/hsa.h>
#include <hsa/hsa_ext_amd.h>
#include <pthread.h>
#include <sched.h>

#include <exception>
#include <new>

#include "mma_engine.h"

namespace mma {

hipError_t launch_transfer(const KernelArgs& args, uint32_t grid, hipStream_t stream);
hipError_t launch_digest(const void* ptr, uint64_t bytes, uint64_t* out, hipStream_t stream);
hipError_t noalloc_setup(int dev);
uint64_t* noalloc_scratch(int dev);
hipError_t launch_noalloc_table(const NoallocTabArgs& t, hipStream_t stream);
hipError_t launch_noalloc(const NoallocArgs& a, uint32_t grid, hipStream_t stream);

namespace {

// ------------------------------------------------------------------ runtime
struct Agents {
  uint32_t want_bdf = 0, want_domain = 0;
  hsa_agent_t gpu{}, cpu{};
  bool have_gpu = false, have_cpu = false;
};

hsa_status_t agent_cb(hsa_agent_t a, void* d) {
  Agents* ag = static_cast<Agents*>(d);
  hsa_device_type_t t;
  if (hsa_agent_get_info(a, HSA_AGENT_INFO_DEVICE, &t) != HSA_STATUS_SUCCESS) return HSA_STATUS_SUCCESS;
  if (t == HSA_DEVICE_TYPE_CPU) {
    if (!ag->have_cpu) {
      ag->cpu = a;
      ag->have_cpu = true;
    }
  } else if (t == HSA_DEVICE_TYPE_GPU) {
    uint32_t bdf = 0, dom = 0;
    hsa_agent_get_info(a, static_cast<hsa_agent_info_t>(HSA_AMD_AGENT_INFO_BDFID), &bdf);
    hsa_agent_get_info(a, static_cast<hsa_agent_info_t>(HSA_AMD_AGENT_INFO_DOMAIN), &dom);
    if (bdf == ag->want_bdf && dom == ag->want_domain && !ag->have_gpu) {
      ag->gpu = a;
      ag->have_gpu = true;
    }
  }
  return HSA_STATUS_SUCCESS;
}

struct StagingCache {  // uncached device memory is kept until process exit
  int dev = -1;
  void* base = nullptr;
  uint64_t bytes = 0;
};
StagingCache g_staging[2];

// ROCr/HIP backend of the engine: records in coherent mapped pinned memory,
// device state in HBM, copy-engine commands through
// hsa_amd_memory_async_copy_on_engine with plain memory signals.
class HsaBackend final : public Backend {
 public:
  HsaBackend(hsa_agent_t gpu, hsa_agent_t cpu) : gpu_(gpu), cpu_(cpu) {}
  mma_status_t alloc_records(uint64_t bytes, void** host, void** dev) override {
    hipError_t e = hipHostMalloc(host, bytes, hipHostMallocMapped | hipHostMallocCoherent);
    if (e != hipSuccess) return fail(MMA_ERR_HIP, "hipHostMalloc(records): %s", hipGetErrorString(e));
    e = hipHostGetDevicePointer(dev, *host, 0);
    if (e != hipSuccess) return fail(MMA_ERR_HIP, "hipHostGetDevicePointer: %s", hipGetErrorString(e));
    return MMA_OK;
  }
  void free_records(void* host) override { (void)hipHostFree(host); }
  mma_status_t alloc_device_state(uint64_t bytes, void** dev) override {
    hipError_t e = hipMalloc(dev, bytes);
    if (e != hipSuccess) return fail(MMA_ERR_HIP, "hipMalloc(device state): %s", hipGetErrorString(e));
    e = hipMemset(*dev, 0, bytes);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) return fail(MMA_ERR_HIP, "hipMemset(device state): %s", hipGetErrorString(e));
    return MMA_OK;
  }
  void free_device_state(void* dev) override { (void)hipFree(dev); }
  mma_status_t alloc_host_scratch(uint64_t bytes, void** host) override {
    if (hipHostMalloc(host, bytes, hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess)
      return fail(MMA_ERR_HIP, "hipHostMalloc(scratch)");
    return MMA_OK;
  }
  void free_host_scratch(void* host) override { (void)hipHostFree(host); }
  // The GPU is the signal's only declared consumer, so ROCr makes it a plain
  // memory signal: no completion interrupt per command (about 3 us of engine
  // time each, measured). The engine thread only polls its value.
  bool signal_create(uint64_t* sig) override {
    hsa_signal_t s;
    if (hsa_amd_signal_create(1, 1, &gpu_, 0, &s) != HSA_STATUS_SUCCESS) return false;
    *sig = s.handle;
    return true;
  }
  void signal_destroy(uint64_t sig) override { hsa_signal_destroy(hsa_signal_t{sig}); }
  void signal_store(uint64_t sig, int64_t v) override { hsa_signal_store_screlease(hsa_signal_t{sig}, v); }
  int64_t signal_load(uint64_t sig) override { return hsa_signal_load_scacquire(hsa_signal_t{sig}); }
  // A signal consumed by GPUs only, whose value a kernel may poll. The value
  // must be the one inside the signal object that the copy engines decrement
  // (the handle is that object's address and the value follows its 8-byte
  // kind); anything else and the copy engines stay out of device control.
  bool signal_create_polled(uint64_t* sig, const int64_t** value) override {
    hsa_signal_t s;
    if (hsa_amd_signal_create(0, 0, nullptr, HSA_AMD_SIGNAL_AMD_GPU_ONLY, &s) != HSA_STATUS_SUCCESS) return false;
    volatile hsa_signal_value_t* v = nullptr;
    if (hsa_amd_signal_value_pointer(s, &v) != HSA_STATUS_SUCCESS || !v ||
        reinterpret_cast<uint64_t>(v) != s.handle + 8) {
      hsa_signal_destroy(s);
      return false;
    }
    *sig = s.handle;
    *value = const_cast<const int64_t*>(reinterpret_cast<volatile int64_t*>(v));
    return true;
  }
  void signal_sub(uint64_t sig, int64_t v) override { hsa_signal_subtract_screlease(hsa_signal_t{sig}, v); }
  bool copy(int engine, void* dst, bool dst_on_device, const void* src, bool src_on_device, uint64_t bytes,
            uint64_t sig) override {
    return hsa_amd_memory_async_copy_on_engine(dst, dst_on_device ? gpu_ : cpu_, src, src_on_device ? gpu_ : cpu_,
                                               bytes, 0, nullptr, hsa_signal_t{sig},
                                               static_cast<hsa_amd_sdma_engine_id_t>(1u << engine),
                                               false) == HSA_STATUS_SUCCESS;
  }
  // hsa_amd_memory_copy_engine_status clears an engine's bit while any copy of
  // this process is on it.
  uint32_t engines_idle(int dir) override {
    uint32_t m = 0;
    if (dir == MMA_H2D)
      hsa_amd_memory_copy_engine_status(gpu_, cpu_, &m);
    else
      hsa_amd_memory_copy_engine_status(cpu_, gpu_, &m);
    return m;
  }

 private:
  hsa_agent_t gpu_, cpu_;
};

struct Runtime {
  int dev = 0;
  mma_config_t ucfg{};
  Config cfg{};
  Agents ag;
  std::unique_ptr<HsaBackend> backend;
  uint32_t wallclock_khz = 100000;
  bool hsa_up = false;
  std::unique_ptr<Engine> eng[2];
  std::mutex submit_mu;
  std::atomic<uint64_t> seq{0};
  Stats stats;
};

Runtime* g_rt = nullptr;
std::mutex g_init_mu;

// Engine threads must not outlive the HIP runtime: if the program exits
// without mma_finalize, they are stopped when this library is unloaded, which
// happens before the runtime it depends on is torn down.
struct ExitGuard {
  ~ExitGuard() {
    std::lock_guard<std::mutex> g(g_init_mu);
    if (!g_rt) return;
    // Transfers still in flight after the wait keep their records and signals:
    // the process is ending, and freeing them could unmap memory that a
    // running kernel still polls.
    for (auto& e : g_rt->eng)
      if (e) e->shutdown(e->wait_idle(2000));
    for (auto& e : g_rt->eng) e.reset();
  }
} g_exit_guard;

void set_affinity_local(pthread_t th, int dev) {
  char bus[64];
  if (hipDeviceGetPCIBusId(bus, sizeof bus, dev) != hipSuccess) return;
  for (char* c = bus; *c; ++c) *c = static_cast<char>(tolower(*c));
  std::string path = std::string("/sys/bus/pci/devices/") + bus + "/local_cpulist";
  FILE* f = fopen(path.c_str(), "r");
  if (!f) return;
  char buf[4096];
  size_t n = fread(buf, 1, sizeof buf - 1, f);
  fclose(f);
  buf[n] = 0;
  cpu_set_t want, have, use;
  CPU_ZERO(&want);
  char* s = buf;
  while (*s) {
    char* end;
    long a = strtol(s, &end, 10);
    if (end == s) break;
    long b = a;
    if (*end == '-') b = strtol(end + 1, &end, 10);
    for (long c = a; c <= b && c < CPU_SETSIZE; ++c) CPU_SET(c, &want);
    s = end;
    while (*s == ',' || *s == '\n' || *s == ' ') ++s;
  }
  if (sched_getaffinity(0, sizeof have, &have) != 0) return;
  CPU_AND(&use, &want, &have);
  if (CPU_COUNT(&use) > 0) pthread_setaffinity_np(th, sizeof use, &use);
}

struct DeviceGuard {
  int prev = -1;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != dev) (void)hipSetDevice(dev);
  }
  ~DeviceGuard() {
    int cur;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

mma_status_t check_ready() {
  if (!g_rt) return fail(MMA_ERR_NOT_INITIALIZED, "mma_init has not been called");
  if (g_sticky.load()) return fail(MMA_ERR_TRANSFER_FAILED, "an earlier transfer failed (sticky; mma_clear_error)");
  return MMA_OK;
}

// [p, p + bytes) must lie inside one allocation: its first and last byte carry
// the same buffer id. (The runtime's RANGE_SIZE attribute is not used: it is
// truncated to 32 bits for allocations of 4 GiB and more.)
bool within_allocation(const void* p, uint64_t bytes) {
  // A range that wraps the address space would put its last byte below p,
  // possibly inside the same allocation.
  const uint64_t span = bytes ? bytes : 1;
  if (span - 1 > UINT64_MAX - reinterpret_cast<uint64_t>(p)) return false;
  uint64_t id0 = 0, id1 = 0;
  hipDeviceptr_t first = const_cast<void*>(p);
  hipDeviceptr_t last = static_cast<uint8_t*>(const_cast<void*>(p)) + (span - 1);
  if (hipPointerGetAttribute(&id0, HIP_POINTER_ATTRIBUTE_BUFFER_ID, first) != hipSuccess ||
      hipPointerGetAttribute(&id1, HIP_POINTER_ATTRIBUTE_BUFFER_ID, last) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return id0 == id1 && id0 != 0;
}

// Allocations validated before, by the runtime's buffer id (unique for the
// life of the process, so an entry can never describe a different live
// allocation): a later range inside one of them needs one attribute query
// instead of three.
class RangeCache {
 public:
  struct Entry {
    uint64_t id = 0, base = 0, size = 0;
    int64_t dev_off = 0;  // host kind: device address - host address
    bool host = false;
  };
  bool find(uint64_t id, bool host, uint64_t p, uint64_t bytes, Entry* out) {
    std::lock_guard<std::mutex> g(mu_);
    for (const Entry& e : e_)
      if (e.id == id && e.host == host && p >= e.base && bytes <= e.size && p - e.base <= e.size - bytes) {
        *out = e;
        return true;
      }
    return false;
  }
  void insert(const Entry& e) {
    std::lock_guard<std::mutex> g(mu_);
    e_[next_++ % kEntries] = e;
  }
  void clear() {
    std::lock_guard<std::mutex> g(mu_);
    for (Entry& e : e_) e = Entry{};
  }

 private:
  static constexpr size_t kEntries = 64;
  std::mutex mu_;
  Entry e_[kEntries];
  size_t next_ = 0;
};
RangeCache g_ranges;

uint64_t buffer_id(const void* p) {
  uint64_t id = 0;
  if (hipPointerGetAttribute(&id, HIP_POINTER_ATTRIBUTE_BUFFER_ID, const_cast<void*>(p)) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  return id;
}

// After a full check of [p, p + bytes): remember the whole allocation.
void remember(uint64_t id, bool host, const void* p, uint64_t bytes, int64_t dev_off) {
  hipDeviceptr_t base = nullptr;
  size_t size = 0;
  if (!id || hipMemGetAddressRange(&base, &size, const_cast<void*>(p)) != hipSuccess) {
    (void)hipGetLastError();
    return;
  }
  const uint64_t b = reinterpret_cast<uint64_t>(base), q = reinterpret_cast<uint64_t>(p);
  if (q < b || bytes > size || q - b > size - bytes) return;  // inconsistent answer: do not rely on it
  RangeCache::Entry e;
  e.id = id;
  e.base = b;
  e.size = size;
  e.dev_off = dev_off;
  e.host = host;
  g_ranges.insert(e);
}

// Pinned, device-mapped host range: returns the device-visible address of p.
// If p is device memory and is_device is given, *is_device is set and
// MMA_ERR_INVALID_ARG returned without an error message.
mma_status_t host_range(const void* p, uint64_t bytes, uint64_t* dev_addr, bool* is_device = nullptr) {
  const uint64_t id = buffer_id(p);
  RangeCache::Entry e;
  if (id && g_ranges.find(id, true, reinterpret_cast<uint64_t>(p), bytes, &e)) {
    *dev_addr = static_cast<uint64_t>(reinterpret_cast<int64_t>(p) + e.dev_off);
    return MMA_OK;
  }
  hipPointerAttribute_t a{};
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return fail(MMA_ERR_NOT_PINNED, "host pointer %p is not pinned host memory", p);
  }
  if (a.type == hipMemoryTypeDevice) {
    if (is_device) {
      *is_device = true;
      return MMA_ERR_INVALID_ARG;
    }
    return fail(MMA_ERR_INVALID_ARG, "%p is device memory, host memory expected", p);
  }
  if (a.type != hipMemoryTypeHost || !a.devicePointer)
    return fail(MMA_ERR_NOT_PINNED, "host pointer %p is not pinned, device-mapped host memory", p);
  if (!within_allocation(p, bytes))
    return fail(MMA_ERR_NOT_PINNED, "host range [%p, +%llu) is not inside one pinned allocation", p,
                static_cast<unsigned long long>(bytes));
  *dev_addr = reinterpret_cast<uint64_t>(a.devicePointer);
  remember(id, true, p, bytes, reinterpret_cast<int64_t>(a.devicePointer) - reinterpret_cast<int64_t>(p));
  return MMA_OK;
}

mma_status_t device_range(const void* p, uint64_t bytes) {
  const uint64_t id = buffer_id(p);
  RangeCache::Entry e;
  if (id && g_ranges.find(id, false, reinterpret_cast<uint64_t>(p), bytes, &e)) return MMA_OK;
  hipPointerAttribute_t a{};
  if (hipPointerGetAttributes(&a, p) != hipSuccess || a.type != hipMemoryTypeDevice) {
    (void)hipGetLastError();
    return fail(MMA_ERR_INVALID_ARG, "%p is not device memory", p);
  }
  if (a.device != g_rt->dev) return fail(MMA_ERR_INVALID_ARG, "%p belongs to device %d", p, a.device);
  if (!within_allocation(p, bytes))
    return fail(MMA_ERR_INVALID_ARG, "device range [%p, +%llu) is not inside one allocation", p,
                static_cast<unsigned long long>(bytes));
  remember(id, false, p, bytes, 0);
  return MMA_OK;
}

// True when nothing can be ordered before work enqueued now on `s`: it is not
// the legacy default stream, it has no pending work, and it either does not
// synchronise with the legacy default stream or that stream is idle too.
// (hipStreamQuery reports hipErrorNotReady for a busy stream; that status is
// not left behind as the thread's last error.)
bool stream_idle(hipStream_t s) {
  if (s == nullptr || s == hipStreamLegacy) return false;
  if (hipStreamQuery(s) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  unsigned int flags = 0;
  if (s != hipStreamPerThread && hipStreamGetFlags(s, &flags) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  if (flags & hipStreamNonBlocking) return true;
  if (hipStreamQuery(nullptr) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return true;
}

// Hand a planned transfer to its engine and enqueue the dummy task on the stream.
//
// The copy must not start before the work that precedes it on the stream, so
// the copy engines normally wait for the dummy kernel's start signal (one
// posted PCIe write, seen by the polling engine thread). When the stream has
// nothing pending, no work precedes the copy: the transfer goes to the engine
// before the launch and the copy engines start while the kernel is still
// being launched. The kernel still holds later stream work until every path
// has landed.
mma_status_t submit(std::unique_ptr<Transfer> x, uint64_t payload_bytes, void* stream, const KvGeom* kv) {
  Runtime* rt = g_rt;
  Engine* e = rt->eng[x->dir].get();
  std::lock_guard<std::mutex> g(rt->submit_mu);
  if (!e->acquire(x.get(), payload_bytes, kv != nullptr, 60000))
    return fail(MMA_ERR_TIMEOUT, "no free transfer record for 60 s");
  static thread_local KernelArgs a;
  const uint64_t wd = static_cast<uint64_t>(rt->cfg.watchdog_ms) * rt->wallclock_khz;
  if (tl_waiter) {
    x->waiter = tl_waiter;
    tl_waiter->submitted = true;
  }
  DeviceGuard dg(rt->dev);
  const hipStream_t hs = static_cast<hipStream_t>(stream);
  if (e->device_control()) {
    // Device control: the transfer is planned in full here and the kernel
    // tracks its completion; no engine-thread work. A transfer with more
    // micro-tasks than a ring holds goes to the engine thread instead.
    const uint32_t grid = x->light >= 0 ? e->prepare(x.get(), ++rt->seq, payload_bytes, kv, wd, a)
                                        : e->prepare_device(x.get(), ++rt->seq, payload_bytes, kv, wd,
                                                            stream_idle(hs), a);
    if (grid) {
      const hipError_t err = launch_transfer(a, grid, hs);
      if (err != hipSuccess) {
        if (x->light >= 0)
          e->release_unused(x.get());
        else
          e->abandon_device(x.get(), rt->cfg.watchdog_ms + 10000ull);
        return fail(MMA_ERR_HIP, "dummy-task kernel launch failed: %s", hipGetErrorString(err));
      }
      e->track(std::move(x));
      return MMA_OK;
    }
  }
  const uint32_t grid = e->prepare(x.get(), ++rt->seq, payload_bytes, kv, wd, a);
  if (!x->self_contained && x->sdma_ok && e->has_sdma() && x->n_claimed < x->tasks.size() && stream_idle(hs)) {
    x->early = true;
    // If the launch fails, the copy engines may already hold part of the
    // transfer: the call returns only after they have drained. A blocking
    // caller's waiter (mma_memcpy_stream) serves for that wait too, so that
    // the caller is still told when the transfer retires.
    if (!x->waiter) x->waiter = std::make_shared<Waiter>();
    std::shared_ptr<Waiter> w = x->waiter;
    Transfer* raw = x.get();  // the engine retires it only after the kernel (or `unlaunched`) releases it
    e->submit(std::move(x));
    const hipError_t err = launch_transfer(a, grid, hs);
    if (err != hipSuccess) {
      raw->unlaunched.store(true, std::memory_order_release);
      std::unique_lock<std::mutex> lk(w->mu);
      w->cv.wait(lk, [&] { return w->done; });
      return fail(MMA_ERR_HIP, "dummy-task kernel launch failed: %s", hipGetErrorString(err));
    }
    return MMA_OK;
  }
  const hipError_t err = launch_transfer(a, grid, hs);
  if (err != hipSuccess) {
    e->release_unused(x.get());
    return fail(MMA_ERR_HIP, "dummy-task kernel launch failed: %s", hipGetErrorString(err));
  }
  // A whole transfer needs nothing from the engine thread but retirement:
  // submitting threads retire it later, and the engine thread is not woken.
  if (x->light >= 0)
    e->track(std::move(x));
  else
    e->submit(std::move(x));
  return MMA_OK;
}

void fill_config(mma_config_t* c, bool use_env) {
  mma_config_t d{};
  d.chunk_bytes = 2 * MiB;
  d.small_bytes = 64 * KiB;
  d.queue_depth = 2;
  d.cu_queue_depth = 4;
  d.cu_workgroups = 16;
  d.cu_sub_bytes = 64 * KiB;
  d.watchdog_ms = 20000;
  d.cu_whole_bytes = static_cast<uint32_t>(kPrefill * kWholeMaxSub);
  d.cu_whole_bytes_d2h = static_cast<uint32_t>(8 * MiB);
  d.control = MMA_CONTROL_HOST;
  d.engine_nap_us = 50;
  if (use_env) {
    d.engine_nap_us = static_cast<uint32_t>(env_u64("MMA_ENGINE_NAP_US", d.engine_nap_us));
    d.control = static_cast<uint32_t>(env_u64("MMA_CONTROL", d.control));
    d.static_cu_percent = static_cast<uint32_t>(env_u64("MMA_STATIC_CU_PERCENT", 0));
    d.duplex_paths_h2d = static_cast<uint32_t>(env_u64("MMA_DUPLEX_PATHS_H2D", 0));
    d.duplex_paths_d2h = static_cast<uint32_t>(env_u64("MMA_DUPLEX_PATHS_D2H", 0));
    d.chunk_bytes = env_u64("MMA_CHUNK_BYTES", d.chunk_bytes);
    d.fallback_bytes = env_u64("MMA_FALLBACK_BYTES", 0);
    d.small_bytes = env_u64("MMA_SMALL_BYTES", d.small_bytes);
    d.queue_depth = static_cast<uint32_t>(env_u64("MMA_QUEUE_DEPTH", d.queue_depth));
    d.cu_queue_depth = static_cast<uint32_t>(env_u64("MMA_CU_QUEUE_DEPTH", d.cu_queue_depth));
    d.backoff_depth = static_cast<uint32_t>(env_u64("MMA_BACKOFF_DEPTH", 0));
    d.path_mask_h2d = static_cast<uint32_t>(env_u64("MMA_PATHS_H2D", 0));
    d.path_mask_d2h = static_cast<uint32_t>(env_u64("MMA_PATHS_D2H", 0));
    d.cu_workgroups = static_cast<uint32_t>(env_u64("MMA_CU_WGS", d.cu_workgroups));
    d.cu_sub_bytes = static_cast<uint32_t>(env_u64("MMA_CU_SUB_BYTES", d.cu_sub_bytes));
    d.watchdog_ms = static_cast<uint32_t>(env_u64("MMA_WATCHDOG_MS", d.watchdog_ms));
    d.sdma_merge_tasks = static_cast<uint32_t>(env_u64("MMA_SDMA_MERGE_TASKS", 0));
    d.cu_whole_bytes = static_cast<uint32_t>(env_u64("MMA_CU_WHOLE_BYTES", d.cu_whole_bytes));
    d.cu_whole_bytes_d2h = static_cast<uint32_t>(env_u64("MMA_CU_WHOLE_BYTES_D2H", d.cu_whole_bytes_d2h));
  }
  *c = d;
}

// No C++ exception may cross the C ABI (a C caller cannot catch it, and it
// would end the process): the entry points that allocate on the host end in a
// handler that turns the exception in flight into a status. Host memory
// exhaustion is MMA_ERR_NO_MEMORY, anything else MMA_ERR_INTERNAL. A call that
// fails this way may have taken a transfer record or light slot it does not
// give back; a later call then waits for another.
void note_exception(mma_status_t s, const char* api, const char* what) noexcept {
  try {
    fail(s, "%s: %s", api, what);
  } catch (...) {
  }
}

mma_status_t boundary_error(const char* api) noexcept {
  try {
    throw;
  } catch (const std::bad_alloc&) {
    note_exception(MMA_ERR_NO_MEMORY, api, "out of host memory");
    return MMA_ERR_NO_MEMORY;
  } catch (const std::exception& e) {
    note_exception(MMA_ERR_INTERNAL, api, e.what());
  } catch (...) {
    note_exception(MMA_ERR_INTERNAL, api, "unknown C++ exception");
  }
  return MMA_ERR_INTERNAL;
}

}  // namespace
}  // namespace mma

using namespace mma;

extern "C" {

mma_status_t mma_config_default(mma_config_t* out) {
  if (!out) return fail(MMA_ERR_INVALID_ARG, "NULL config");
  fill_config(out, false);
  return MMA_OK;
}

mma_status_t mma_init(int hip_device, const mma_config_t* user_cfg) try {
  std::lock_guard<std::mutex> g(g_init_mu);
  if (g_rt) return fail(MMA_ERR_ALREADY_INITIALIZED, "already initialised");
  g_ranges.clear();  // device entries were checked against the previous device
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || hip_device < 0 || hip_device >= ndev) {
    (void)hipGetLastError();
    return fail(MMA_ERR_INVALID_ARG, "invalid HIP device %d (%d devices)", hip_device, ndev);
  }
  // Zero selects a field's default, whether it came in the caller's
  // configuration or from the environment (where an unparsable value reads
  // as 0).
  mma_config_t c, d;
  fill_config(&d, false);
  if (user_cfg)
    c = *user_cfg;
  else
    fill_config(&c, true);
  if (!c.chunk_bytes) c.chunk_bytes = d.chunk_bytes;
  if (!c.small_bytes) c.small_bytes = d.small_bytes;
  if (!c.queue_depth) c.queue_depth = d.queue_depth;
  if (!c.cu_queue_depth) c.cu_queue_depth = d.cu_queue_depth;
  if (!c.cu_workgroups) c.cu_workgroups = d.cu_workgroups;
  if (!c.cu_sub_bytes) c.cu_sub_bytes = d.cu_sub_bytes;
  if (!c.watchdog_ms) c.watchdog_ms = d.watchdog_ms;
  if (!c.cu_whole_bytes) c.cu_whole_bytes = d.cu_whole_bytes;
  if (!c.cu_whole_bytes_d2h) c.cu_whole_bytes_d2h = d.cu_whole_bytes_d2h;
  if (!c.engine_nap_us) c.engine_nap_us = d.engine_nap_us;
  if (!c.fallback_bytes) c.fallback_bytes = 2 * c.chunk_bytes;
  // A micro-task's ring entries must fit the ring next to the end-marker
  // reserve of one slot per wave (counted without forming chunk + sub, which
  // could wrap).
  if (c.cu_sub_bytes % 16 || c.cu_sub_bytes < 256 || c.chunk_bytes % 16 || c.queue_depth > 16 ||
      c.cu_workgroups > kMaxWorkgroups || c.cu_queue_depth > 64 ||
      (c.engine_nap_us > 1000 && c.engine_nap_us != MMA_ENGINE_NAP_OFF) ||
      c.chunk_bytes / c.cu_sub_bytes + (c.chunk_bytes % c.cu_sub_bytes != 0) > kRingSize / 2)
    return fail(MMA_ERR_INVALID_ARG, "invalid configuration");
  if (c.static_cu_percent > 100) return fail(MMA_ERR_INVALID_ARG, "static_cu_percent > 100");
  if (c.control > MMA_CONTROL_DEVICE) return fail(MMA_ERR_INVALID_ARG, "unknown control mode %u", c.control);

  std::unique_ptr<Runtime> rt(new Runtime());
  rt->dev = hip_device;
  DeviceGuard dg(hip_device);
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, hip_device) != hipSuccess) return fail(MMA_ERR_HIP, "hipGetDeviceProperties");
  int wclk = 0;
  if (hipDeviceGetAttribute(&wclk, hipDeviceAttributeWallClockRate, hip_device) == hipSuccess && wclk > 0)
    rt->wallclock_khz = static_cast<uint32_t>(wclk);
  if (hsa_init() != HSA_STATUS_SUCCESS) return fail(MMA_ERR_HSA, "hsa_init failed");
  // Every way out of this call but success (an error return, an exception)
  // gives the ROCr reference back, after the engines (their threads and
  // signals) are gone.
  struct HsaRef {
    Runtime* rt;
    bool held = true;
    ~HsaRef() {
      if (!held) return;
      rt->eng[0].reset();
      rt->eng[1].reset();
      hsa_shut_down();
    }
  } hsa_ref{rt.get()};
  rt->hsa_up = true;
  rt->ag.want_bdf = static_cast<uint32_t>((prop.pciBusID << 8) | (prop.pciDeviceID << 3));
  rt->ag.want_domain = static_cast<uint32_t>(prop.pciDomainID);
  hsa_iterate_agents(agent_cb, &rt->ag);
  if (!rt->ag.have_gpu || !rt->ag.have_cpu) {
    return fail(MMA_ERR_HSA, "no ROCr agent for HIP device %d", hip_device);
  }
  uint32_t avail[2] = {0, 0}, nsdma = 0;
  hsa_amd_memory_copy_engine_status(rt->ag.gpu, rt->ag.cpu, &avail[MMA_H2D]);
  hsa_amd_memory_copy_engine_status(rt->ag.cpu, rt->ag.gpu, &avail[MMA_D2H]);
  hsa_agent_get_info(rt->ag.gpu, static_cast<hsa_agent_info_t>(HSA_AMD_AGENT_INFO_NUM_SDMA_ENG), &nsdma);
  const uint32_t host_facing = nsdma >= 16 ? 0xFFFFu : ((1u << nsdma) - 1u);
  uint32_t mask[2] = {c.path_mask_h2d, c.path_mask_d2h};
  const bool mask_given[2] = {c.path_mask_h2d != 0, c.path_mask_d2h != 0};
  for (int d = 0; d < 2; ++d) {
    if (!mask[d]) mask[d] = MMA_PATH_CU | (avail[d] & host_facing);
    mask[d] = (mask[d] & MMA_PATH_CU) | (mask[d] & avail[d] & 0xFFFFu);
    if (!(mask[d] & 0xFFFFu)) mask[d] |= MMA_PATH_CU;  // some path must carry the work
  }
  c.path_mask_h2d = mask[0];
  c.path_mask_d2h = mask[1];
  // Paths while the other direction moves (see Engine::set_peer). A static
  // split fixes each micro-task's path at plan time, so it keeps its masks.
  uint32_t duplex[2] = {c.duplex_paths_h2d, c.duplex_paths_d2h};
  for (int d = 0; d < 2; ++d) {
    if (c.static_split || duplex[d] == MMA_DUPLEX_UNCHANGED) {
      duplex[d] = mask[d];
      continue;
    }
    // Default: the direction's engines without the CU path; for device-to-host
    // with the default path mask, engines 2-5 instead of the host-facing ones.
    if (!duplex[d]) duplex[d] = d == MMA_H2D || mask_given[d] ? (mask[d] & 0xFFFFu) : 0x3Cu;
    duplex[d] = (duplex[d] & mask[d] & MMA_PATH_CU) | (duplex[d] & avail[d] & 0xFFFFu);
    if (!duplex[d]) duplex[d] = mask[d];
  }
  c.duplex_paths_h2d = duplex[0];
  c.duplex_paths_d2h = duplex[1];
  // Back-off depth: given, it applies to every path; by default each path
  // pulls again as soon as it is below its own queue depth.
  const uint32_t backoff_given = c.backoff_depth;
  if (!c.backoff_depth) c.backoff_depth = c.queue_depth;
  rt->ucfg = c;
  Config& k = rt->cfg;
  k.chunk = c.chunk_bytes;
  k.fallback = c.fallback_bytes;
  k.small = c.small_bytes;
  k.sub = c.cu_sub_bytes;
  k.depth = c.queue_depth;
  k.cu_depth = c.cu_queue_depth;
  k.backoff = c.backoff_depth;
  k.cu_backoff = backoff_given;
  k.cu_wgs = c.cu_workgroups;
  k.watchdog_ms = c.watchdog_ms;
  k.mask[0] = mask[0];
  k.mask[1] = mask[1];
  k.duplex[0] = duplex[0];
  k.duplex[1] = duplex[1];
  k.device = c.control == MMA_CONTROL_DEVICE ? 1u : 0u;
  k.device_cu_percent = c.static_cu_percent ? c.static_cu_percent : kDeviceCuPercent;
  k.static_split = c.static_split;
  k.static_cu_percent = c.static_cu_percent;
  k.whole[MMA_H2D] = c.cu_whole_bytes;
  k.whole[MMA_D2H] = c.cu_whole_bytes_d2h;
  k.nap_ns = c.engine_nap_us == MMA_ENGINE_NAP_OFF ? 0 : 1000ull * c.engine_nap_us;
  k.merge = c.sdma_merge_tasks ? c.sdma_merge_tasks
                              : static_cast<uint32_t>(std::max<uint64_t>(1, 64 * MiB / c.chunk_bytes));

  // SDMA staging for the KV kinds: one chunk per SDMA slot, in uncached device
  // memory (coherent between the copy engines and every XCD's L2 without
  // cache maintenance). Kept for the process lifetime and reused.
  const uint64_t stage_bytes = (std::max<uint64_t>(k.chunk, 2 * MiB) + 4095) & ~4095ull;
  for (int d = 0; d < 2; ++d) {
    const uint32_t n = static_cast<uint32_t>(__builtin_popcount((mask[d] | duplex[d]) & 0xFFFFu));
    const uint64_t need = n * k.depth * stage_bytes;
    StagingCache& sc = g_staging[d];
    if (need && (sc.dev != hip_device || sc.bytes < need)) {
      void* p = nullptr;
      if (hipExtMallocWithFlags(&p, need, hipDeviceMallocUncached) != hipSuccess) {
        (void)hipGetLastError();
        return fail(MMA_ERR_HIP, "staging allocation of %llu bytes failed", static_cast<unsigned long long>(need));
      }
      sc.dev = hip_device;
      sc.base = p;
      sc.bytes = need;
    }
  }
  // The no-alloc KV fetch's scratch array: its address on this device, looked
  // up once with the device current.
  {
    const hipError_t e = noalloc_setup(hip_device);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return fail(MMA_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    }
  }
  rt->backend.reset(new HsaBackend(rt->ag.gpu, rt->ag.cpu));
  for (int d = 0; d < 2; ++d) {
    rt->eng[d].reset(new Engine(d, k, rt->backend.get(), &rt->stats));
    const uint32_t engines = (mask[d] | duplex[d]) & 0xFFFFu;
    mma_status_t s = rt->eng[d]->init(engines, stage_bytes, engines ? g_staging[d].base : nullptr);
    if (s != MMA_OK) return s;  // hsa_ref stops the engines created so far
    set_affinity_local(rt->eng[d]->native_handle(), hip_device);
  }
  rt->eng[MMA_D2H]->set_peer(rt->eng[MMA_H2D].get());
  rt->eng[MMA_H2D]->set_peer(rt->eng[MMA_D2H].get());
  if (env_u64("MMA_TRACE", 0)) g_trace = 1;
  hsa_ref.held = false;  // mma_finalize gives it back
  g_rt = rt.release();
  return MMA_OK;
} catch (...) {
  return boundary_error("mma_init");
}

mma_status_t mma_finalize(void) try {
  std::lock_guard<std::mutex> g(g_init_mu);
  if (!g_rt) return fail(MMA_ERR_NOT_INITIALIZED, "not initialised");
  bool drained = true;
  for (auto& e : g_rt->eng) drained = e->wait_idle(30000) && drained;
  if (!drained) return fail(MMA_ERR_TIMEOUT, "in-flight transfers did not drain");
  {
    DeviceGuard dg(g_rt->dev);
    // each engine thread reads the other engine's counters: stop both before freeing either
    for (auto& e : g_rt->eng) e->shutdown();
    for (auto& e : g_rt->eng) e.reset();
  }
  if (g_rt->hsa_up) hsa_shut_down();
  delete g_rt;
  g_rt = nullptr;
  return MMA_OK;
} catch (...) {
  return boundary_error("mma_finalize");
}

mma_status_t mma_get_config(mma_config_t* out) {
  if (!out) return fail(MMA_ERR_INVALID_ARG, "NULL config");
  if (!g_rt) return fail(MMA_ERR_NOT_INITIALIZED, "not initialised");
  *out = g_rt->ucfg;
  return MMA_OK;
}

mma_status_t mma_synchronize(uint32_t timeout_ms) try {
  if (!g_rt) return fail(MMA_ERR_NOT_INITIALIZED, "not initialised");
  for (auto& e : g_rt->eng)
    if (!e->wait_idle(timeout_ms)) return fail(MMA_ERR_TIMEOUT, "transfers still in flight");
  return g_sticky.load() ? fail(MMA_ERR_TRANSFER_FAILED, "a transfer failed") : MMA_OK;
} catch (...) {
  return boundary_error("mma_synchronize");
}

mma_status_t mma_host_alloc(uint64_t bytes, void** out) {
  if (!out) return fail(MMA_ERR_INVALID_ARG, "NULL out");
  *out = nullptr;
  if (!bytes) return MMA_OK;
  int dev = g_rt ? g_rt->dev : 0;
  DeviceGuard dg(dev);
  hipError_t e = hipHostMalloc(out, bytes, hipHostMallocMapped | hipHostMallocCoherent);
  if (e != hipSuccess) {
    *out = nullptr;
    return fail(MMA_ERR_NO_MEMORY, "hipHostMalloc(%llu): %s", static_cast<unsigned long long>(bytes),
                hipGetErrorString(e));
  }
  return MMA_OK;
}

mma_status_t mma_host_free(void* p) {
  if (!p) return MMA_OK;
  hipError_t e = hipHostFree(p);
  return e == hipSuccess ? MMA_OK : fail(MMA_ERR_HIP, "hipHostFree: %s", hipGetErrorString(e));
}

mma_status_t mma_memcpy_async(void* dst, const void* src, uint64_t bytes, int32_t dir, void* stream) {
  mma_status_t s = check_ready();
  if (s) return s;
  if (dir != MMA_H2D && dir != MMA_D2H) return fail(MMA_ERR_INVALID_ARG, "dir must be MMA_H2D or MMA_D2H");
  if (!bytes) return MMA_OK;
  if (!dst || !src) return fail(MMA_ERR_INVALID_ARG, "NULL pointer with bytes > 0");
  mma_copy_desc_t d{dst, src, bytes};
  return mma_weights_load(&d, 1, dir, stream);
}

mma_status_t mma_memcpy_stream(void* dst, const void* src, uint64_t bytes, int32_t dir, void* stream,
                               int32_t* outcome) try {
  if (outcome) *outcome = MMA_COPY_NOT_ENQUEUED;
  std::shared_ptr<Waiter> w = std::make_shared<Waiter>();
  tl_waiter = w;
  mma_status_t s = mma_memcpy_async(dst, src, bytes, dir, stream);
  tl_waiter.reset();
  if (s) return s;  // refused; or a failed launch, after which nothing of the copy is in flight
  if (!w->submitted) {  // nothing to move
    if (outcome) *outcome = MMA_COPY_RETIRED;
    return MMA_OK;
  }
  if (outcome) *outcome = MMA_COPY_IN_FLIGHT;
  {
    DeviceGuard dg(g_rt->dev);
    const hipError_t e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(MMA_ERR_HIP, "hipStreamSynchronize: %s", hipGetErrorString(e));
  }
  // The stream has passed the dummy task; the engine thread retires the
  // transfer right after (or this thread does, for a transfer the submitting
  // threads track), which is when its outcome is final.
  Engine* e = g_rt->eng[dir].get();
  std::unique_lock<std::mutex> lk(w->mu);
  const auto deadline = std::chrono::steady_clock::now() +
                        std::chrono::milliseconds(static_cast<uint64_t>(g_rt->cfg.watchdog_ms) + 10000);
  while (!w->done) {
    if (std::chrono::steady_clock::now() >= deadline) return fail(MMA_ERR_TIMEOUT, "copy not retired");
    lk.unlock();
    e->reap();
    lk.lock();
    if (!w->done) w->cv.wait_for(lk, std::chrono::microseconds(20));
  }
  if (outcome) *outcome = MMA_COPY_RETIRED;
  return w->failed ? fail(MMA_ERR_TRANSFER_FAILED, "the copy failed") : MMA_OK;
} catch (...) {
  return boundary_error("mma_memcpy_stream");
}

mma_status_t mma_memcpy(void* dst, const void* src, uint64_t bytes, int32_t dir) {
  return mma_memcpy_stream(dst, src, bytes, dir, nullptr, nullptr);
}

mma_status_t mma_weights_load(const mma_copy_desc_t* list, uint64_t n, int32_t dir, void* stream) try {
  const uint64_t t_api = now_ns();
  mma_status_t s = check_ready();
  if (s) return s;
  if (dir != MMA_H2D && dir != MMA_D2H) return fail(MMA_ERR_INVALID_ARG, "dir must be MMA_H2D or MMA_D2H");
  if (!n) return MMA_OK;
  if (!list) return fail(MMA_ERR_INVALID_ARG, "NULL list");
  Runtime* rt = g_rt;
  DeviceGuard dg(rt->dev);
  std::vector<uint64_t> sizes(n), src_cu(n), dst_cu(n);
  std::vector<std::pair<uint64_t, uint64_t>> dsts;
  uint64_t total = 0;
  for (uint64_t i = 0; i < n; ++i) {
    const mma_copy_desc_t& d = list[i];
    sizes[i] = d.bytes;
    if (!d.bytes) continue;
    if (!d.dst || !d.src) return fail(MMA_ERR_INVALID_ARG, "list[%llu]: NULL pointer", (unsigned long long)i);
    const void* host = dir == MMA_H2D ? d.src : d.dst;
    const void* dev = dir == MMA_H2D ? d.dst : d.src;
    uint64_t hdev = 0;
    if ((s = host_range(host, d.bytes, &hdev))) return s;
    if ((s = device_range(dev, d.bytes))) return s;
    src_cu[i] = dir == MMA_H2D ? hdev : reinterpret_cast<uint64_t>(d.src);
    dst_cu[i] = dir == MMA_H2D ? reinterpret_cast<uint64_t>(d.dst) : hdev;
    dsts.push_back({reinterpret_cast<uint64_t>(d.dst), reinterpret_cast<uint64_t>(d.dst) + d.bytes});
    total += d.bytes;
  }
  if (!total) return MMA_OK;
  if (!ranges_disjoint(dsts)) return fail(MMA_ERR_INVALID_ARG, "destination ranges overlap");
  std::unique_ptr<Transfer> x = make_list_transfer(dir, list, n, sizes.data(), src_cu.data(), dst_cu.data(), rt->cfg);
  // Device control plans a transfer into one ring of kRingSize micro-tasks. A
  // copy or list with more is planned again at twice the chunk size until it
  // fits, rather than handed to the engine thread (the model wake-up list has
  // 7,723 micro-tasks at 2 MiB, 3,890 at 4 MiB). A list of more tensors than
  // that never fits (each tensor is at least one micro-task) and is not
  // planned again.
  if (rt->cfg.device && dsts.size() <= kRingSize) {
    Config c = rt->cfg;
    while (x->tasks.size() > kRingSize && c.chunk < kDeviceMaxChunk) {
      c.chunk *= 2;
      x = make_list_transfer(dir, list, n, sizes.data(), src_cu.data(), dst_cu.data(), c);
    }
  }
  x->t_api = t_api;
  return submit(std::move(x), total, stream, nullptr);
} catch (...) {
  return boundary_error("mma_weights_load");
}

// A validated KV call: geometry handed to the kernels, and where the pool is.
struct KvCall {
  KvGeom kv;
  uint64_t piece = 0, slot_bytes = 0;
  uint32_t ppb = 0;
  uint64_t pool_cu = 0;  // the pool's device-visible address
  bool pool_dev = false; // the pool is device memory of this GPU
};

typedef bool (*tables_check_fn)(const int32_t* src, uint32_t src_count, const int32_t* dst, uint32_t dst_count,
                                uint64_t n);

// Validation shared by the KV calls (nothing enqueued): layout, GPU block
// layout geometry, tables (in range, distinct destinations), the pool (pinned
// host memory, or device memory of this GPU) and the layer tensors. n > 0 and
// the library initialised.
static mma_status_t kv_check(const mma_kv_layout_t* lay, const void* host_pool, const void* const* layers,
                             const int32_t* host_slots, const int32_t* gpu_blocks, uint64_t n, int dir,
                             tables_check_fn tables, KvCall* out) {
  mma_status_t s;
  if (!lay || !host_pool || !layers || !host_slots || !gpu_blocks)
    return fail(MMA_ERR_INVALID_ARG, "NULL argument");
  KvSizes sz;
  if (!kv_sizes(lay->num_layers, lay->block_tokens, lay->kv_heads, lay->head_dim, lay->elem_bytes,
                lay->gpu_num_blocks, lay->host_num_slots, kMaxLayers, &sz))
    return fail(MMA_ERR_INVALID_ARG, "invalid KV layout: a field is 0, more than %u layers, a piece above 4 GiB, "
                                     "or a pool or layer size beyond 64 bits", kMaxLayers);
  const uint64_t piece = sz.piece;
  KvGeom& kv = out->kv;
  kv.layout = lay->gpu_layout;
  if (lay->gpu_layout == MMA_KV_LAYOUT_XPACKED) {
    // One wave stages whole heads of one piece in LDS: the tile must hold at
    // least one head's rows (with 16 bytes of padding per row) in every
    // staging order the kernel uses.
    const uint64_t E = lay->elem_bytes, B = lay->block_tokens, R = static_cast<uint64_t>(lay->head_dim) * E;
    if ((E != 1 && E != 2 && E != 4 && E != 8) || R % 16 || (B * E) % 16)
      return fail(MMA_ERR_INVALID_ARG, "x-packed KV layout needs elem_bytes in {1,2,4,8} and head_dim*elem_bytes, "
                                       "block_tokens*elem_bytes multiples of 16");
    const uint64_t need = std::max({B * (R + 16), (R / 16) * (B * 16 + 16), (R / E) * (B * E + 16)});
    const uint64_t lds_wave = std::max<uint64_t>(need, 16 * KiB);
    if (need > kMaxLdsPerWave)
      return fail(MMA_ERR_INVALID_ARG, "x-packed KV layout: one head of one block needs %llu bytes of LDS (max %llu)",
                  static_cast<unsigned long long>(need), static_cast<unsigned long long>(kMaxLdsPerWave));
    if ((reinterpret_cast<uintptr_t>(host_pool) & 15u) != 0)
      return fail(MMA_ERR_INVALID_ARG, "x-packed KV layout needs a 16-byte-aligned pool");
    kv.tokens = lay->block_tokens;
    kv.heads = lay->kv_heads;
    kv.row_bytes = static_cast<uint32_t>(R);
    kv.elem = lay->elem_bytes;
    kv.lds_wave = static_cast<uint32_t>((lds_wave + 15) & ~15ull);
  } else if (lay->gpu_layout == MMA_KV_LAYOUT_HND) {
    // Rows of head_dim elements move whole, in 16-byte units.
    const uint64_t R = static_cast<uint64_t>(lay->head_dim) * lay->elem_bytes;
    if (R % 16)
      return fail(MMA_ERR_INVALID_ARG, "head-major KV layout needs head_dim*elem_bytes a multiple of 16");
    if ((reinterpret_cast<uintptr_t>(host_pool) & 15u) != 0)
      return fail(MMA_ERR_INVALID_ARG, "head-major KV layout needs a 16-byte-aligned pool");
    kv.tokens = lay->block_tokens;
    kv.heads = lay->kv_heads;
    kv.row_bytes = static_cast<uint32_t>(R);
    kv.elem = lay->elem_bytes;
  } else if (lay->gpu_layout != MMA_KV_LAYOUT_PIECE) {
    return fail(MMA_ERR_INVALID_ARG, "unknown GPU KV layout %u", lay->gpu_layout);
  }
  const uint32_t ppb = 2 * lay->num_layers;
  const uint64_t slot_bytes = sz.slot, pool_bytes = sz.pool, layer_bytes = sz.layer;
  bool ok = dir == MMA_H2D ? tables(host_slots, lay->host_num_slots, gpu_blocks, lay->gpu_num_blocks, n)
                           : tables(gpu_blocks, lay->gpu_num_blocks, host_slots, lay->host_num_slots, n);
  if (!ok) return fail(MMA_ERR_INVALID_ARG, "block table entry out of range or duplicate destination");
  // The pool is pinned host memory, or device memory of this GPU (a KV tier
  // in HBM): then the transfer is an HBM gather/scatter carried by the CU path.
  uint64_t pool_cu = 0;
  bool pool_dev = false;
  s = host_range(host_pool, pool_bytes, &pool_cu, &pool_dev);
  if (pool_dev) {
    s = device_range(host_pool, pool_bytes);
    pool_cu = reinterpret_cast<uint64_t>(host_pool);
  }
  if (s) return s;
  kv.layers = lay->num_layers;
  kv.piece = piece;
  kv.kstride = piece * lay->gpu_num_blocks;
  for (uint32_t l = 0; l < lay->num_layers; ++l) {
    if (!layers[l]) return fail(MMA_ERR_INVALID_ARG, "NULL layer pointer %u", l);
    if ((s = device_range(layers[l], layer_bytes))) return s;
    if (kv.layout != MMA_KV_LAYOUT_PIECE && (reinterpret_cast<uintptr_t>(layers[l]) & 15u) != 0)
      return fail(MMA_ERR_INVALID_ARG, "x-packed and head-major KV layouts need 16-byte-aligned layer tensors "
                                       "(layer %u)", l);
    kv.layer_ptr[l] = reinterpret_cast<uint64_t>(layers[l]);
  }
  out->piece = piece;
  out->slot_bytes = slot_bytes;
  out->ppb = ppb;
  out->pool_cu = pool_cu;
  out->pool_dev = pool_dev;
  return MMA_OK;
}

static mma_status_t kv_common(const mma_kv_layout_t* lay, const void* host_pool, const void* const* layers,
                              const int32_t* host_slots, const int32_t* gpu_blocks, uint64_t n, int dir,
                              void* stream) try {
  const uint64_t t_api = now_ns();
  mma_status_t s = check_ready();
  if (s) return s;
  if (!n) return MMA_OK;
  Runtime* rt = g_rt;
  DeviceGuard dg(rt->dev);
  KvCall c;
  if ((s = kv_check(lay, host_pool, layers, host_slots, gpu_blocks, n, dir, tables_valid, &c))) return s;
  const uint64_t per_task = std::max<uint64_t>(rt->cfg.chunk / c.piece, 1) * c.piece;
  const bool sdma_ok = per_task <= rt->eng[dir]->stage_bytes() && !c.pool_dev;
  std::unique_ptr<Transfer> x = make_kv_transfer(dir, c.piece, c.ppb, reinterpret_cast<uint64_t>(host_pool),
                                                 c.pool_cu, c.pool_dev, sdma_ok, host_slots, gpu_blocks, n, rt->cfg);
  // A pool in HBM, GPU blocks in the piece or the head-major layout: one
  // launch of the pool kernel sized to the bytes, if the table finds room
  // (acquire). x-packed blocks need the LDS transform of the ring path.
  x->pool_launch = c.pool_dev && (c.kv.layout == MMA_KV_LAYOUT_PIECE || c.kv.layout == MMA_KV_LAYOUT_HND);
  x->t_api = t_api;
  return submit(std::move(x), n * c.slot_bytes, stream, &c.kv);
} catch (...) {
  return boundary_error("mma_kv_fetch/mma_kv_offload");
}

// Table check of the no-alloc KV fetch: the same rule as tables_valid, with
// fixed storage instead of a buffer per call (a bitmap over destination
// blocks, cleared again after use, or a sorted copy for very large caches).
std::mutex g_noalloc_mu;
constexpr uint32_t kNoallocBitmapBits = 1u << 24;
uint64_t g_noalloc_seen[kNoallocBitmapBits / 64];
int32_t g_noalloc_sorted[kNoallocMaxBlocks];

bool noalloc_tables_valid(const int32_t* src, uint32_t src_count, const int32_t* dst, uint32_t dst_count,
                          uint64_t n) {
  if (n > kNoallocMaxBlocks) return false;
  for (uint64_t i = 0; i < n; ++i) {
    if (src[i] < 0 || static_cast<uint32_t>(src[i]) >= src_count) return false;
    if (dst[i] < 0 || static_cast<uint32_t>(dst[i]) >= dst_count) return false;
  }
  std::lock_guard<std::mutex> g(g_noalloc_mu);
  if (dst_count <= kNoallocBitmapBits) {
    uint64_t i = 0;
    bool ok = true;
    for (; i < n; ++i) {
      uint64_t& w = g_noalloc_seen[static_cast<uint32_t>(dst[i]) >> 6];
      const uint64_t bit = 1ull << (static_cast<uint32_t>(dst[i]) & 63u);
      if (w & bit) {
        ok = false;
        break;
      }
      w |= bit;
    }
    for (uint64_t j = 0; j < i; ++j) g_noalloc_seen[static_cast<uint32_t>(dst[j]) >> 6] = 0;
    return ok;
  }
  std::copy(dst, dst + n, g_noalloc_sorted);
  std::sort(g_noalloc_sorted, g_noalloc_sorted + n);
  return std::adjacent_find(g_noalloc_sorted, g_noalloc_sorted + n) == g_noalloc_sorted + n;
}

mma_status_t mma_kv_fetch(const mma_kv_layout_t* layout, const void* host_pool, void* const* gpu_layers,
                          const int32_t* host_slots, const int32_t* gpu_blocks, uint64_t n_blocks, void* stream) {
  return kv_common(layout, host_pool, const_cast<const void* const*>(gpu_layers), host_slots, gpu_blocks, n_blocks,
                   MMA_H2D, stream);
}

mma_status_t mma_kv_offload(const mma_kv_layout_t* layout, void* host_pool, const void* const* gpu_layers,
                            const int32_t* gpu_blocks, const int32_t* host_slots, uint64_t n_blocks, void* stream) {
  return kv_common(layout, host_pool, gpu_layers, host_slots, gpu_blocks, n_blocks, MMA_D2H, stream);
}

mma_status_t mma_kv_fetch_noalloc(const mma_kv_layout_t* layout, const void* host_pool, void* const* gpu_layers,
                                  const int32_t* host_slots, const int32_t* gpu_blocks, uint64_t n_blocks,
                                  void* stream) try {
  mma_status_t s = check_ready();
  if (s) return s;
  if (!n_blocks) return MMA_OK;
  if (n_blocks > kNoallocMaxBlocks)
    return fail(MMA_ERR_INVALID_ARG, "mma_kv_fetch_noalloc: %llu blocks in one call, at most %u (its fixed table)",
                static_cast<unsigned long long>(n_blocks), kNoallocMaxBlocks);
  Runtime* rt = g_rt;
  DeviceGuard dg(rt->dev);
  uint64_t* scratch = noalloc_scratch(rt->dev);
  if (!scratch) return fail(MMA_ERR_NOT_INITIALIZED, "no scratch array address for device %d", rt->dev);
  KvCall c;
  if ((s = kv_check(layout, host_pool, const_cast<const void* const*>(gpu_layers), host_slots, gpu_blocks, n_blocks,
                    MMA_H2D, noalloc_tables_valid, &c)))
    return s;
  NoallocArgs a;
  memset(&a, 0, sizeof a);
  a.scratch = scratch;
  a.pool = c.pool_cu;
  a.slot_bytes = c.slot_bytes;
  a.piece = c.piece;
  a.kstride = c.kv.kstride;
  a.ppb = c.ppb;
  a.units = n_blocks * c.ppb;
  a.per_claim = static_cast<uint32_t>(std::max<uint64_t>(1, rt->cfg.sub / c.piece));
  a.layout = c.kv.layout;
  a.tokens = c.kv.tokens;
  a.heads = c.kv.heads;
  a.row_bytes = c.kv.row_bytes;
  a.elem = c.kv.elem;
  a.lds_wave = c.kv.lds_wave;
  memcpy(a.layer_ptr, c.kv.layer_ptr, sizeof(uint64_t) * c.kv.layers);
  const hipStream_t hs = static_cast<hipStream_t>(stream);
  // The table goes into the scratch array through kernel arguments, chunk by
  // chunk, on the caller's stream: no copy call and no staging buffer.
  NoallocTabArgs t;
  memset(&t, 0, offsetof(NoallocTabArgs, e));
  t.scratch = scratch;
  for (uint64_t first = 0; first < n_blocks; first += kNoallocTabChunk) {
    const uint32_t count = static_cast<uint32_t>(std::min<uint64_t>(kNoallocTabChunk, n_blocks - first));
    t.first = static_cast<uint32_t>(first);
    t.count = count;
    t.reset = first == 0 ? 1u : 0u;
    for (uint32_t j = 0; j < count; ++j)
      t.e[j] = static_cast<uint64_t>(static_cast<uint32_t>(host_slots[first + j])) |
               (static_cast<uint64_t>(static_cast<uint32_t>(gpu_blocks[first + j])) << 32);
    const hipError_t err = launch_noalloc_table(t, hs);
    if (err != hipSuccess) return fail(MMA_ERR_HIP, "no-alloc table launch failed: %s", hipGetErrorString(err));
  }
  // CU path alone: the engine thread's workgroup limit for a transfer over
  // PCIe (1.5x for the transformed layouts); a pool in HBM gets a grid sized
  // for HBM rates.
  const uint64_t claims = (a.units + a.per_claim - 1) / a.per_claim;
  const uint64_t wgs = c.kv.layout == MMA_KV_LAYOUT_PIECE ? rt->cfg.cu_wgs : (3ull * rt->cfg.cu_wgs + 1) / 2;
  const uint64_t cap = c.pool_dev ? 2048 : std::min<uint64_t>(wgs, kMaxWorkgroups);
  const uint32_t grid =
      static_cast<uint32_t>(std::max<uint64_t>(1, std::min<uint64_t>((claims + kWavesPerWG - 1) / kWavesPerWG, cap)));
  const hipError_t err = launch_noalloc(a, grid, hs);
  return err == hipSuccess ? MMA_OK : fail(MMA_ERR_HIP, "no-alloc KV fetch launch failed: %s", hipGetErrorString(err));
} catch (...) {
  return boundary_error("mma_kv_fetch_noalloc");
}

mma_status_t mma_digest_u32(const void* dev_ptr, uint64_t bytes, uint64_t* dev_out, void* stream) {
  if (!g_rt) return fail(MMA_ERR_NOT_INITIALIZED, "not initialised");
  if (!bytes) return MMA_OK;
  if (!dev_ptr || !dev_out) return fail(MMA_ERR_INVALID_ARG, "NULL pointer");
  if (reinterpret_cast<uintptr_t>(dev_ptr) & 3u) return fail(MMA_ERR_INVALID_ARG, "dev_ptr must be 4-byte aligned");
  if (reinterpret_cast<uintptr_t>(dev_out) & 7u) return fail(MMA_ERR_INVALID_ARG, "dev_out must be 8-byte aligned");
  mma_status_t s;
  DeviceGuard dg(g_rt->dev);
  if ((s = device_range(dev_ptr, bytes))) return s;
  if ((s = device_range(dev_out, 8))) return s;
  hipError_t e = launch_digest(dev_ptr, bytes, dev_out, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MMA_OK : fail(MMA_ERR_HIP, "digest launch: %s", hipGetErrorString(e));
}

mma_status_t mma_get_stats(mma_stats_t* out) try {
  if (!out) return fail(MMA_ERR_INVALID_ARG, "NULL out");
  if (!g_rt) return fail(MMA_ERR_NOT_INITIALIZED, "not initialised");
  // Transfers that the submitting threads track are retired when a thread
  // reaps: do it here, so the figures cover every transfer whose kernel is done.
  for (auto& e : g_rt->eng) e->reap();
  memset(out, 0, sizeof *out);
  Stats& st = g_rt->stats;
  out->transfers = st.transfers;
  out->failed_transfers = st.failed;
  for (int i = 0; i < MMA_NUM_PATHS; ++i) {
    out->path_bytes[i] = st.path_bytes[i];
    out->path_tasks[i] = st.path_tasks[i];
  }
  out->staging_bytes = st.staging_bytes;
  out->sdma_submit_failures = st.submit_failures;
  out->engine_wall_busy_ns = st.busy_ns;
  out->sdma_foreign_busy_skips = st.foreign_skips;
  out->sdma_commands = st.sdma_commands;
  out->pool_launches = st.pool_launches;
  out->engine_naps = st.naps;
  out->sdma_congestion_backoffs = st.congestion_backoffs;
  uint64_t cpu = 0;
  for (auto& e : g_rt->eng) {
    clockid_t cid;
    timespec ts;
    if (pthread_getcpuclockid(e->native_handle(), &cid) == 0 && clock_gettime(cid, &ts) == 0)
      cpu += static_cast<uint64_t>(ts.tv_sec) * 1000000000ull + ts.tv_nsec;
  }
  out->engine_cpu_ns = cpu;
  out->sdma_engines_h2d = g_rt->eng[MMA_H2D]->sdma_mask();
  out->sdma_engines_d2h = g_rt->eng[MMA_D2H]->sdma_mask();
  out->cu_path_enabled = (g_rt->eng[MMA_H2D]->cu_enabled() ? 1u : 0u) | (g_rt->eng[MMA_D2H]->cu_enabled() ? 2u : 0u);
  return MMA_OK;
} catch (...) {
  return boundary_error("mma_get_stats");
}

mma_status_t mma_reset_stats(void) {
  if (!g_rt) return fail(MMA_ERR_NOT_INITIALIZED, "not initialised");
  g_rt->stats.reset();
  return MMA_OK;
}

const char* mma_status_str(mma_status_t s) {
  switch (s) {
    case MMA_OK: return "MMA_OK";
    case MMA_ERR_NOT_INITIALIZED: return "MMA_ERR_NOT_INITIALIZED";
    case MMA_ERR_INVALID_ARG: return "MMA_ERR_INVALID_ARG";
    case MMA_ERR_NOT_PINNED: return "MMA_ERR_NOT_PINNED";
    case MMA_ERR_HIP: return "MMA_ERR_HIP";
    case MMA_ERR_HSA: return "MMA_ERR_HSA";
    case MMA_ERR_TRANSFER_FAILED: return "MMA_ERR_TRANSFER_FAILED";
    case MMA_ERR_ALREADY_INITIALIZED: return "MMA_ERR_ALREADY_INITIALIZED";
    case MMA_ERR_NO_MEMORY: return "MMA_ERR_NO_MEMORY";
    case MMA_ERR_BUFFER_TOO_SMALL: return "MMA_ERR_BUFFER_TOO_SMALL";
    case MMA_ERR_TIMEOUT: return "MMA_ERR_TIMEOUT";
    case MMA_ERR_INTERNAL: return "MMA_ERR_INTERNAL";
    default: return "MMA_ERR_UNKNOWN";
  }
}

const char* mma_last_error(void) { return t_err.c_str(); }

mma_status_t mma_clear_error(void) {
  g_sticky.store(0);
  t_err.clear();
  return MMA_OK;
}

mma_status_t mma_trace_enable(int32_t on) try {
  std::lock_guard<std::mutex> g(g_trace_mu);
  if (on && !g_trace.load()) g_trace_buf.clear();
  g_trace = on ? 1 : 0;
  return MMA_OK;
} catch (...) {
  return boundary_error("mma_trace_enable");
}

mma_status_t mma_trace_read(mma_trace_rec_t* out, uint64_t cap, uint64_t* n_out) try {
  if (!n_out || (cap && !out)) return fail(MMA_ERR_INVALID_ARG, "NULL argument");
  if (g_rt)
    for (auto& e : g_rt->eng) e->reap();  // records of tracked transfers are written when they retire
  std::lock_guard<std::mutex> g(g_trace_mu);
  const uint64_t n = std::min<uint64_t>(cap, g_trace_buf.size());
  for (uint64_t i = 0; i < n; ++i) out[i] = g_trace_buf[i];
  g_trace_buf.erase(g_trace_buf.begin(), g_trace_buf.begin() + static_cast<long>(n));
  *n_out = n;
  return MMA_OK;
} catch (...) {
  return boundary_error("mma_trace_read");
}

mma_status_t mma_test_set_fault(int32_t kind, uint64_t value) {
  switch (kind) {
    case MMA_FAULT_ENGINE_STALL_US: g_fault_stall_us = value; return MMA_OK;
    case MMA_FAULT_SDMA_SUBMIT_FAIL: g_fault_submit_fail = value; return MMA_OK;
    case MMA_FAULT_ENGINE_IGNORE: g_fault_ignore = value; return MMA_OK;
    case MMA_FAULT_DEVICE_SIGNAL_HOLD: g_fault_signal_hold = value; return MMA_OK;
    case MMA_FAULT_POOL_NO_TABLE: g_fault_pool_no_table = value; return MMA_OK;
    default: return fail(MMA_ERR_INVALID_ARG, "unknown fault kind %d", kind);
  }
}

}  // extern "C"
