// Host side of the multipath copy path: the C ABI, the per-direction engine
// threads (Section 4: separate H2D and D2H engine instances), SDMA submission
// through ROCr, and the CU-ring bookkeeping shared with the dummy-task kernel.
//
// Roles, mapped to the paper's components (Section 3, Figure "Overview"):
//   Transfer Task Interceptor -> the mma_* entry points: record the request,
//                                plan it, enqueue the dummy task on the stream.
//   Sync Engine               -> the record's started/complete words and the
//                                dummy-task kernel's wait (mma_kernels.hip).
//   Task Manager              -> plan_list / plan_kv (mma_plan.cpp) + per-task
//                                completion accounting here.
//   Path Selector             -> Engine::pull_cu / Engine::pull_sdma: every path
//                                pulls the next micro-task only while its
//                                outstanding queue has room (backpressure).
//   Task Launcher             -> SDMA: hsa_amd_memory_async_copy_on_engine;
//                                CU path: ring entries consumed by the kernel.
#include <hip/hip_runtime.h>
#include <hsa/hsa.h>
#include <hsa/hsa_ext_amd.h>
#include <pthread.h>
#include <sched.h>
#include <time.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <deque>
#include <memory>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "../../include/mma.h"
#include "mma_plan.h"
#include "mma_proto.h"

namespace mma {

hipError_t launch_transfer(const KernelArgs& args, uint32_t grid, hipStream_t stream);
hipError_t launch_digest(const void* ptr, uint64_t bytes, uint64_t* out, hipStream_t stream);

namespace {

// ------------------------------------------------------------------ utilities
thread_local std::string t_err;

mma_status_t fail(mma_status_t s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  t_err = buf;
  return s;
}

uint64_t now_ns() {
  timespec ts;
  clock_gettime(CLOCK_MONOTONIC, &ts);
  return static_cast<uint64_t>(ts.tv_sec) * 1000000000ull + ts.tv_nsec;
}

template <class T>
inline T ld_acq(const T* p) {
  return __atomic_load_n(p, __ATOMIC_ACQUIRE);
}
template <class T>
inline void st_rel(T* p, T v) {
  __atomic_store_n(p, v, __ATOMIC_RELEASE);
}

inline void cpu_relax() { __builtin_ia32_pause(); }

uint64_t env_u64(const char* name, uint64_t dflt) {
  const char* v = getenv(name);
  if (!v || !*v) return dflt;
  return strtoull(v, nullptr, 0);
}

constexpr uint64_t KiB = 1024, MiB = 1024 * 1024;
constexpr uint64_t kSmallSub = 16 * KiB;  // one wave register batch

// ------------------------------------------------------------------ transfer
enum class Kind : uint8_t { kLinear, kKvFetch, kKvOffload };

// Completion slot of one synchronous call (mma_memcpy): set by the engine
// thread when it retires the transfer.
struct Waiter {
  std::mutex mu;
  std::condition_variable cv;
  bool submitted = false, done = false, failed = false;
};
thread_local std::shared_ptr<Waiter> tl_waiter;

struct Task {
  uint64_t src_dma, dst_dma;  // addresses used by the SDMA engines (linear kinds)
  uint64_t src_cu, dst_cu;    // addresses used by CU loads/stores (linear kinds)
  uint64_t host_dma, host_cu; // KV: contiguous host range of the task's pieces
  uint64_t bytes;             // linear: bytes; KV: pieces
  uint64_t blk;               // KV: GPU block index
  uint32_t p0;                // KV: first piece (2*l + k)
  uint32_t flags;             // kPlanCuOnly
};

struct Transfer {
  uint64_t seq = 0;
  int dir = MMA_H2D;
  Kind kind = Kind::kLinear;
  uint32_t rec_idx = 0;
  Record* rec = nullptr;      // host address of the shared record
  std::vector<Task> tasks;
  std::vector<uint8_t> claimed;
  std::vector<uint32_t> left;  // CU entries outstanding per CU-path task
  size_t cur_cu = 0, cur_sdma = 0, n_claimed = 0, n_done = 0;
  uint64_t piece = 0;
  bool sdma_ok = true;         // SDMA may carry this transfer's tasks
  // CU ring bookkeeping
  uint64_t pushed = 0, done_upto = 0;
  uint32_t waves = 0;          // waves of the dummy-task kernel
  bool pool_dev = false;       // KV pool in device memory: HBM gather/scatter, one entry per task
  bool self_contained = false; // whole transfer in the kernel args; the kernel does not wait on the host
  uint64_t sub = 0;            // bytes per CU ring entry of a linear transfer
  std::shared_ptr<Waiter> waiter;  // set for synchronous calls
  int32_t owner[kRingSize];    // >= 0: CU-path task; < 0: -(1 + SDMA slot id)
  uint8_t tdone[kRingSize];
  uint32_t cu_busy = 0;
  bool cu_full = false;
  int sdma_cu_pending = 0;     // SDMA slots that will still append ring entries
  int sdma_refs = 0;           // SDMA slots referencing this transfer
  uint64_t heartbeat = 0;
  uint64_t bytes = 0;          // payload bytes
  // trace timestamps (CLOCK_MONOTONIC ns)
  uint64_t t_api = 0, t_submit = 0, t_started = 0, t_first_sdma = 0, t_last_task = 0, t_complete = 0;
  uint64_t path_tasks[MMA_NUM_PATHS] = {};
  bool started = false, closed = false, completed = false, failed = false, ignored = false, aborting = false;
  bool progress = false;
};

// ------------------------------------------------------------------ engine
enum SlotState : int {
  kFree = 0,
  kCopy,            // SDMA: linear micro-task in flight
  kH2DStage,        // SDMA: host slot range -> staging
  kH2DScatterPush,  // waiting for ring room to append the staging scatter
  kH2DScatter,      // CU: staging -> paged layout
  kD2HGatherPush,   // waiting for ring room to append the staging gather
  kD2HGather,       // CU: paged layout -> staging
  kD2HStage,        // SDMA: staging -> host slot range
};

struct SdmaSlot {
  hsa_signal_t sig{};
  int state = kFree;
  Transfer* x = nullptr;
  size_t task = 0, task_end = 0;  // micro-tasks [task, task_end) carried by this slot's command
  uint64_t count = 0;     // their total: bytes (linear) or pieces (KV, one block's run)
  uint32_t left = 0;      // ring entries outstanding
  uint64_t staging = 0;   // device address of this slot's staging buffer
  int path = 0;
  uint64_t t_submit = 0;  // current copy-engine command: submission time and size
  uint64_t op_bytes = 0;
};

struct SdmaPath {
  int engine = 0;
  std::vector<int> slots;  // slot ids
  int busy = 0;
  bool full = false;
  bool congested = false;  // a command is long overdue: pull nothing more until the engine drains
};

struct Config {
  uint64_t chunk, fallback, small, sub;
  uint32_t depth, cu_depth, backoff, cu_wgs, watchdog_ms;
  uint32_t mask[2];
  uint32_t static_split, static_cu_percent;
  uint32_t merge;       // max micro-tasks per copy-engine command
};

struct Stats {
  std::atomic<uint64_t> transfers{0}, failed{0}, staging_bytes{0}, submit_failures{0}, busy_ns{0};
  std::atomic<uint64_t> foreign_skips{0}, congestion_backoffs{0}, sdma_commands{0};
  std::atomic<uint64_t> path_bytes[MMA_NUM_PATHS], path_tasks[MMA_NUM_PATHS];
  Stats() {
    for (auto& v : path_bytes) v = 0;
    for (auto& v : path_tasks) v = 0;
  }
  void reset() {
    transfers = failed = staging_bytes = submit_failures = busy_ns = foreign_skips = congestion_backoffs = 0;
    sdma_commands = 0;
    for (auto& v : path_bytes) v = 0;
    for (auto& v : path_tasks) v = 0;
  }
};

std::atomic<int> g_sticky{0};

// Per-transfer trace records (MMA_TRACE=1 or mma_trace_enable): a bounded ring.
std::atomic<int> g_trace{0};
std::mutex g_trace_mu;
std::deque<mma_trace_rec_t> g_trace_buf;
constexpr size_t kTraceCap = 65536;
std::atomic<uint64_t> g_fault_stall_us{0}, g_fault_submit_fail{0}, g_fault_ignore{0};

class Engine {
 public:
  Engine(int dir, const Config& cfg, hsa_agent_t gpu, hsa_agent_t cpu, Stats* st)
      : dir_(dir), cfg_(cfg), gpu_(gpu), cpu_(cpu), st_(st) {}
  ~Engine() { shutdown(); }

  mma_status_t init(uint32_t sdma_mask, uint64_t stage_bytes, void* staging_base) {
    hipError_t e = hipHostMalloc(reinterpret_cast<void**>(&recs_), sizeof(Record) * kRecords,
                                 hipHostMallocMapped | hipHostMallocCoherent);
    if (e != hipSuccess) return fail(MMA_ERR_HIP, "hipHostMalloc(records): %s", hipGetErrorString(e));
    memset(recs_, 0, sizeof(Record) * kRecords);
    e = hipHostGetDevicePointer(reinterpret_cast<void**>(&recs_dev_), recs_, 0);
    if (e != hipSuccess) return fail(MMA_ERR_HIP, "hipHostGetDevicePointer: %s", hipGetErrorString(e));
    e = hipMalloc(reinterpret_cast<void**>(&ds_), sizeof(DevState) * kRecords);
    if (e != hipSuccess) return fail(MMA_ERR_HIP, "hipMalloc(device state): %s", hipGetErrorString(e));
    e = hipMemset(ds_, 0, sizeof(DevState) * kRecords);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) return fail(MMA_ERR_HIP, "hipMemset(device state): %s", hipGetErrorString(e));
    for (uint32_t i = 0; i < kRecords; ++i) free_recs_.push_back(i);
    stage_bytes_ = stage_bytes;
    uint8_t* stage = static_cast<uint8_t*>(staging_base);
    for (int eng = 0; eng < MMA_MAX_SDMA; ++eng) {
      if (!(sdma_mask & (1u << eng))) continue;
      SdmaPath p;
      p.engine = eng;
      for (uint32_t d = 0; d < cfg_.depth; ++d) {
        SdmaSlot s;
        // The GPU is the signal's only declared consumer, so ROCr makes it a
        // plain memory signal: no completion interrupt per command (about 3 us
        // of engine time each, measured). This thread only polls its value.
        if (hsa_amd_signal_create(1, 1, &gpu_, 0, &s.sig) != HSA_STATUS_SUCCESS)
          return fail(MMA_ERR_HSA, "hsa_amd_signal_create failed");
        s.staging = stage ? reinterpret_cast<uint64_t>(stage) : 0;
        if (stage) stage += stage_bytes;
        s.path = static_cast<int>(paths_.size());
        p.slots.push_back(static_cast<int>(slots_.size()));
        slots_.push_back(s);
      }
      paths_.push_back(p);
    }
    mma_status_t w = warm_up();
    if (w != MMA_OK) return w;
    thread_ = std::thread([this] { loop(); });
    return MMA_OK;
  }

  // The first command on an engine makes ROCr create that engine's queue
  // (milliseconds); do it here rather than inside the first transfer.
  mma_status_t warm_up() {
    if (paths_.empty()) return MMA_OK;
    void* host = nullptr;
    if (hipHostMalloc(&host, 4096, hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess)
      return fail(MMA_ERR_HIP, "hipHostMalloc(warm-up)");
    mma_status_t rc = MMA_OK;
    for (auto& path : paths_) {
      SdmaSlot& s = slots_[path.slots[0]];
      hsa_signal_store_screlease(s.sig, 1);
      const auto eng = static_cast<hsa_amd_sdma_engine_id_t>(1u << path.engine);
      hsa_status_t r = dir_ == MMA_H2D
          ? hsa_amd_memory_async_copy_on_engine(reinterpret_cast<void*>(s.staging), gpu_, host, cpu_, 4096, 0,
                                                nullptr, s.sig, eng, false)
          : hsa_amd_memory_async_copy_on_engine(host, cpu_, reinterpret_cast<void*>(s.staging), gpu_, 4096, 0,
                                                nullptr, s.sig, eng, false);
      if (r != HSA_STATUS_SUCCESS) {
        rc = fail(MMA_ERR_HSA, "SDMA engine %d rejected a warm-up copy", path.engine);
        break;
      }
      const uint64_t t0 = now_ns();
      hsa_signal_value_t v;
      while ((v = hsa_signal_load_scacquire(s.sig)) > 0 && now_ns() - t0 < 10000000000ull) cpu_relax();
      if (v != 0) {  // still in flight or failed: leave the engine out rather than reuse its signal
        rc = fail(MMA_ERR_HSA, "SDMA engine %d did not complete a warm-up copy", path.engine);
        break;
      }
    }
    (void)hipHostFree(host);
    return rc;
  }

  void shutdown() {
    {
      std::lock_guard<std::mutex> g(mu_);
      if (!thread_.joinable()) return;
      stop_ = true;
      stop_flag_ = true;
    }
    cv_.notify_all();
    thread_.join();
    for (auto& s : slots_) hsa_signal_destroy(s.sig);
    slots_.clear();
    if (ds_) (void)hipFree(ds_);
    if (recs_) (void)hipHostFree(recs_);
    ds_ = nullptr;
    recs_ = nullptr;
  }

  pthread_t native_handle() { return thread_.native_handle(); }
  uint32_t sdma_mask() const {
    uint32_t m = 0;
    for (auto& p : paths_) m |= 1u << p.engine;
    return m;
  }
  bool cu_enabled() const { return (cfg_.mask[dir_] & MMA_PATH_CU) != 0; }
  bool has_sdma() const { return !paths_.empty(); }
  uint64_t stage_bytes() const { return stage_bytes_; }

  // Blocks until a record is free (or the timeout passes). Called with the
  // submission mutex held, never by the engine thread.
  bool acquire_record(Transfer* x, uint64_t timeout_ms) {
    std::unique_lock<std::mutex> lk(mu_);
    if (!cv_done_.wait_for(lk, std::chrono::milliseconds(timeout_ms), [&] { return !free_recs_.empty(); }))
      return false;
    x->rec_idx = free_recs_.front();
    free_recs_.pop_front();
    x->rec = &recs_[x->rec_idx];
    return true;
  }
  void release_record_unused(Transfer* x) {
    std::lock_guard<std::mutex> g(mu_);
    free_recs_.push_back(x->rec_idx);
    cv_done_.notify_all();
  }
  Record* rec_dev(uint32_t i) const { return recs_dev_ + i; }
  DevState* ds(uint32_t i) const { return ds_ + i; }

  // CU path's first pulls, made before the transfer is handed to the engine
  // thread (no concurrent access to x yet): the dummy task's workers can start
  // copying as soon as the stream reaches them, without a host round trip.
  void prefill(Transfer* x) { pull_cu(x); }

  void submit(std::unique_ptr<Transfer> x) {
    {
      std::lock_guard<std::mutex> g(mu_);
      incoming_.push_back(std::move(x));
      ++inflight_;
    }
    n_incoming_.fetch_add(1, std::memory_order_release);
    cv_.notify_all();
  }

  bool wait_idle(uint64_t timeout_ms) {
    std::unique_lock<std::mutex> lk(mu_);
    return cv_done_.wait_for(lk, std::chrono::milliseconds(timeout_ms), [&] { return inflight_ == 0; });
  }

 private:
  // ---------------------------------------------------------------- ring
  // Append the ring entries of one unit of work. `a` is the contiguous side
  // (linear: source; KV: host or staging range), `b` the other side (linear:
  // destination; KV: GPU block). Returns the number appended, 0 if no room.
  uint32_t push_unit(Transfer* x, int32_t owner, uint32_t kind, uint64_t a, uint64_t b, uint64_t count,
                     uint32_t p0) {
    uint64_t per, ne;
    if ((kind & kEntryKindMask) == kEntryCopy) {
      per = x->sub;
    } else {
      // A wave's ring entry carries cu_sub_bytes of pieces across PCIe; for an
      // HBM-resident pool (latency ~1 us instead of several) a whole micro-task.
      per = x->pool_dev ? count : std::max<uint64_t>(1, cfg_.sub / x->piece);
    }
    ne = (count + per - 1) / per;
    // Keep one slot per wave free for the end markers written at close.
    if (x->pushed + ne - x->done_upto > kRingSize - x->waves) return 0;
    Record* r = x->rec;
    for (uint64_t k = 0; k < ne; ++k) {
      const uint64_t t = x->pushed++;
      const uint32_t slot = static_cast<uint32_t>(t % kRingSize);
      const uint64_t c = std::min(per, count - k * per);
      CuEntry* e = &r->ring[slot];
      if ((kind & kEntryKindMask) == kEntryCopy) {
        e->a = a + k * per;
        e->b = b + k * per;
        e->kind_p0 = kind;
      } else {
        e->a = a + k * per * x->piece;
        e->b = b;
        e->kind_p0 = kind | ((p0 + static_cast<uint32_t>(k * per)) << 8);
      }
      e->count = static_cast<uint32_t>(c);
      x->owner[slot] = owner;
      x->tdone[slot] = 0;
      // Payload first, then both tags: a reader that sees either tag also sees
      // the payload written before it (x86 stores are ordered).
      const uint64_t tag = make_tag(x->seq, t);
      st_rel(&e->tag0, tag);
      st_rel(&e->tag1, tag);
    }
    return static_cast<uint32_t>(ne);
  }

  void task_done(Transfer* x, size_t i, int path_stat) {
    ++x->n_done;
    ++x->path_tasks[path_stat];
    if (x->n_done == x->tasks.size()) x->t_last_task = now_ns();
    const Task& t = x->tasks[i];
    const uint64_t bytes = x->kind == Kind::kLinear ? t.bytes : t.bytes * x->piece;
    st_->path_bytes[path_stat] += bytes;
    st_->path_tasks[path_stat] += 1;
    x->progress = true;
  }

  bool scan_cu(Transfer* x) {
    bool p = false;
    Record* r = x->rec;
    for (uint64_t t = x->done_upto; t < x->pushed; ++t) {
      const uint32_t slot = static_cast<uint32_t>(t % kRingSize);
      if (x->tdone[slot]) continue;
      if (ld_acq(&r->done[slot]) != make_tag(x->seq, t)) continue;
      x->tdone[slot] = 1;
      p = true;
      const int32_t own = x->owner[slot];
      if (own >= 0) {
        if (--x->left[own] == 0) {
          --x->cu_busy;
          task_done(x, static_cast<size_t>(own), MMA_NUM_PATHS - 1);
        }
      } else {
        // Staging step of an SDMA slot; ignore it if the slot was released
        // early because the transfer was aborted.
        SdmaSlot& s = slots_[-own - 1];
        if (s.x == x && (s.state == kH2DScatter || s.state == kD2HGather) && --s.left == 0) sdma_cu_stage_done(s);
      }
    }
    while (x->done_upto < x->pushed && x->tdone[x->done_upto % kRingSize]) ++x->done_upto;
    return p;
  }

  // ---------------------------------------------------------------- CU path
  bool pull_cu(Transfer* x) {
    if (x->failed || x->ignored || x->aborting) return false;
    const bool any = cu_enabled() || x->pool_dev;
    // An HBM-resident pool keeps every wave busy: two micro-tasks per wave outstanding.
    const uint32_t depth = x->pool_dev ? 2 * x->waves : cfg_.cu_depth;
    bool p = false;
    while (true) {
      if (x->cu_busy >= depth) x->cu_full = true;
      if (x->cu_full && x->cu_busy < std::min(cfg_.backoff, depth)) x->cu_full = false;
      if (x->cu_full) break;
      size_t i = x->cur_cu;
      while (i < x->tasks.size() && (x->claimed[i] || (x->tasks[i].flags & kPlanSdmaOnly) ||
                                      (!any && !(x->tasks[i].flags & kPlanCuOnly))))
        ++i;
      x->cur_cu = i;
      if (i >= x->tasks.size()) break;
      const Task& t = x->tasks[i];
      uint32_t ne;
      if (x->kind == Kind::kLinear)
        ne = push_unit(x, static_cast<int32_t>(i), kEntryCopy, t.src_cu, t.dst_cu, t.bytes, 0);
      else
        ne = push_unit(x, static_cast<int32_t>(i), x->kind == Kind::kKvFetch ? kEntryToPaged : kEntryFromPaged,
                       t.host_cu, t.blk, t.bytes, t.p0);
      if (!ne) break;
      x->claimed[i] = 1;
      ++x->n_claimed;
      x->left[i] = ne;
      ++x->cu_busy;
      p = true;
    }
    return p;
  }

  // ---------------------------------------------------------------- SDMA path
  bool sdma_copy(SdmaSlot& s, void* dst, hsa_agent_t dst_agent, const void* src, hsa_agent_t src_agent,
                 uint64_t bytes) {
    uint64_t f = g_fault_submit_fail.load();
    while (f > 0) {
      if (g_fault_submit_fail.compare_exchange_weak(f, f - 1)) return false;
    }
    if (!s.x->t_first_sdma) s.x->t_first_sdma = now_ns();
    s.t_submit = now_ns();
    s.op_bytes = bytes;
    hsa_signal_store_screlease(s.sig, 1);
    const hsa_status_t r = hsa_amd_memory_async_copy_on_engine(
        dst, dst_agent, src, src_agent, bytes, 0, nullptr, s.sig,
        static_cast<hsa_amd_sdma_engine_id_t>(1u << paths_[s.path].engine), false);
    if (r == HSA_STATUS_SUCCESS) st_->sdma_commands += 1;
    return r == HSA_STATUS_SUCCESS;
  }

  void free_slot(SdmaSlot& s) {
    SdmaPath& p = paths_[s.path];
    --p.busy;
    if (s.x) --s.x->sdma_refs;
    s.state = kFree;
    s.x = nullptr;
  }

  // The staged CU step of an SDMA-carried KV micro-task has landed.
  void slot_tasks_done(SdmaSlot& s) {
    for (size_t i = s.task; i < s.task_end; ++i) task_done(s.x, i, paths_[s.path].engine);
  }

  void sdma_cu_stage_done(SdmaSlot& s) {
    Transfer* x = s.x;
    const Task& t = x->tasks[s.task];
    if (s.state == kH2DScatter) {
      st_->staging_bytes += s.count * x->piece;
      slot_tasks_done(s);
      free_slot(s);
    } else if (s.state == kD2HGather) {
      st_->staging_bytes += s.count * x->piece;
      if (sdma_copy(s, reinterpret_cast<void*>(t.host_dma), cpu_, reinterpret_cast<void*>(s.staging), gpu_,
                    s.count * x->piece)) {
        s.state = kD2HStage;
      } else {
        // The gathered bytes are in staging and cannot reach the host this way.
        st_->submit_failures += 1;
        x->failed = true;
        slot_tasks_done(s);
        free_slot(s);
      }
    }
  }

  bool try_push_stage(SdmaSlot& s) {
    Transfer* x = s.x;
    const Task& t = x->tasks[s.task];
    const int32_t own = -1 - static_cast<int32_t>(&s - slots_.data());
    uint32_t ne;
    if (s.state == kH2DScatterPush)
      ne = push_unit(x, own, kEntryToPaged | kEntryAcquire, s.staging, t.blk, s.count, t.p0);
    else
      ne = push_unit(x, own, kEntryFromPaged, s.staging, t.blk, s.count, t.p0);
    if (!ne) return false;
    s.left = ne;
    s.state = s.state == kH2DScatterPush ? kH2DScatter : kD2HGather;
    --x->sdma_cu_pending;
    return true;
  }

  bool poll_sdma() {
    bool p = false;
    for (auto& s : slots_) {
      if (s.state == kH2DScatterPush || s.state == kD2HGatherPush) {
        if (s.x->aborting) {
          --s.x->sdma_cu_pending;
          free_slot(s);
          p = true;
        } else if (try_push_stage(s)) {
          s.x->progress = true;
          p = true;
        }
        continue;
      }
      if (s.state == kH2DScatter || s.state == kD2HGather) {
        if (s.x->aborting) {  // the kernel has left; its ring entries will never run
          free_slot(s);
          p = true;
        }
        continue;
      }
      if (s.state != kCopy && s.state != kH2DStage && s.state != kD2HStage) continue;
      const hsa_signal_value_t v = hsa_signal_load_scacquire(s.sig);
      if (v > 0) continue;
      p = true;
      Transfer* x = s.x;
      x->progress = true;
      if (v < 0) {
        x->failed = true;
        if (s.state == kH2DStage) --x->sdma_cu_pending;
        slot_tasks_done(s);
        free_slot(s);
        continue;
      }
      if (s.state == kCopy || s.state == kD2HStage) {
        slot_tasks_done(s);
        free_slot(s);
      } else {  // kH2DStage landed: scatter it on the CU side
        s.state = kH2DScatterPush;
        if (x->aborting) {
          --x->sdma_cu_pending;
          free_slot(s);
        } else {
          try_push_stage(s);
        }
      }
    }
    return p;
  }

  // Next SDMA-eligible task of the oldest started transfer.
  bool next_sdma_task(Transfer*& out, size_t& idx) {
    for (auto& up : active_) {
      Transfer* x = up.get();
      if (!x->started || x->failed || x->ignored || x->aborting || !x->sdma_ok) continue;
      size_t i = x->cur_sdma;
      while (i < x->tasks.size() && (x->claimed[i] || (x->tasks[i].flags & kPlanCuOnly))) ++i;
      x->cur_sdma = i;
      if (i < x->tasks.size()) {
        out = x;
        idx = i;
        return true;
      }
    }
    return false;
  }

  // One copy-engine command carries the claimed micro-task i and the unclaimed
  // ones that directly follow it in both address spaces (a linear run, or one
  // KV block's consecutive pieces that fit the staging slot), up to cfg.merge.
  // Each ROCr copy command costs about 8 us of engine time (measured), so at
  // small chunk sizes one command per micro-task would cap an engine well
  // below the link.
  size_t merge_run(const Transfer* x, size_t i) const {
    const bool sdma_only = (x->tasks[i].flags & kPlanSdmaOnly) != 0;
    uint64_t total = x->tasks[i].bytes;
    size_t j = i + 1;
    for (; j < x->tasks.size() && j - i < cfg_.merge; ++j) {
      const Task& a = x->tasks[j - 1];
      const Task& b = x->tasks[j];
      if (x->claimed[j] || (b.flags & kPlanCuOnly) || ((b.flags & kPlanSdmaOnly) != 0) != sdma_only) break;
      if (x->kind == Kind::kLinear) {
        if (b.src_dma != a.src_dma + a.bytes || b.dst_dma != a.dst_dma + a.bytes) break;
      } else {
        if (b.blk != a.blk || b.p0 != a.p0 + a.bytes || b.host_dma != a.host_dma + a.bytes * x->piece ||
            (total + b.bytes) * x->piece > stage_bytes_)
          break;
      }
      total += b.bytes;
    }
    return j;
  }

  // A copy-engine command is overdue when it has been in flight for four times
  // what its size needs at 50 GB/s, plus 0.5 ms of slack.
  bool overdue(const SdmaPath& path, uint64_t now) const {
    for (int id : path.slots) {
      const SdmaSlot& s = slots_[id];
      if (s.state != kCopy && s.state != kH2DStage && s.state != kD2HStage) continue;
      if (now - s.t_submit > 4 * s.op_bytes / 50 + 500000) return true;  // ns
    }
    return false;
  }

  // Paths that can make progress take work (Section 2.2; Section 3.4 contention
  // back-off). ROCr keeps one in-order command queue per engine per process, so
  // a command placed behind another component's copies waits for all of them:
  // an engine that ROCr reports in use while none of our commands is on it is
  // busy with foreign work and is skipped; an engine with an overdue command is
  // backed off until it drains.
  bool pull_sdma() {
    bool p = false;
    const uint32_t bo = std::min(cfg_.backoff, cfg_.depth);
    uint32_t free_mask = 0;
    bool have_mask = false;
    const uint64_t now = now_ns();
    for (size_t k = 0; k < paths_.size(); ++k) {
      SdmaPath& path = paths_[(k + rr_) % paths_.size()];
      if (path.congested) {
        if (path.busy > 0) continue;
        path.congested = false;
      } else if (path.busy > 0 && overdue(path, now)) {
        path.congested = true;
        st_->congestion_backoffs += 1;
        continue;
      }
      if (path.busy == 0) {
        if (!have_mask) {
          if (dir_ == MMA_H2D)
            hsa_amd_memory_copy_engine_status(gpu_, cpu_, &free_mask);
          else
            hsa_amd_memory_copy_engine_status(cpu_, gpu_, &free_mask);
          have_mask = true;
        }
        if (!(free_mask & (1u << path.engine))) {
          st_->foreign_skips += 1;
          continue;
        }
      }
      for (int id : path.slots) {
        if (path.busy >= static_cast<int>(cfg_.depth)) path.full = true;
        if (path.full && path.busy < static_cast<int>(bo)) path.full = false;
        if (path.full) break;
        SdmaSlot& s = slots_[id];
        if (s.state != kFree) continue;
        Transfer* x;
        size_t i;
        if (!next_sdma_task(x, i)) return p;
        const Task& t = x->tasks[i];
        const size_t end = merge_run(x, i);
        for (size_t j = i; j < end; ++j) x->claimed[j] = 1;
        x->n_claimed += end - i;
        s.x = x;
        s.task = i;
        s.task_end = end;
        s.count = 0;
        for (size_t j = i; j < end; ++j) s.count += x->tasks[j].bytes;
        ++path.busy;
        ++x->sdma_refs;
        bool ok = true;
        if (x->kind == Kind::kLinear) {
          const bool h2d = dir_ == MMA_H2D;
          ok = sdma_copy(s, reinterpret_cast<void*>(t.dst_dma), h2d ? gpu_ : cpu_,
                         reinterpret_cast<void*>(t.src_dma), h2d ? cpu_ : gpu_, s.count);
          s.state = kCopy;
        } else if (x->kind == Kind::kKvFetch) {
          ok = sdma_copy(s, reinterpret_cast<void*>(s.staging), gpu_, reinterpret_cast<void*>(t.host_dma), cpu_,
                         s.count * x->piece);
          s.state = kH2DStage;
          if (ok) ++x->sdma_cu_pending;
        } else {
          s.state = kD2HGatherPush;
          ++x->sdma_cu_pending;
          try_push_stage(s);
        }
        if (!ok) {
          // Re-route: the tasks go back to the queue, CU path only.
          st_->submit_failures += 1;
          for (size_t j = i; j < end; ++j) {
            x->claimed[j] = 0;
            x->tasks[j].flags = (x->tasks[j].flags & ~kPlanSdmaOnly) | kPlanCuOnly;
          }
          x->n_claimed -= end - i;
          x->cur_cu = std::min(x->cur_cu, i);
          free_slot(s);
        }
        x->progress = true;
        p = true;
      }
    }
    ++rr_;
    return p;
  }

  // ---------------------------------------------------------------- lifecycle
  bool advance(Transfer* x) {
    Record* r = x->rec;
    bool p = false;
    if (!x->started && !x->ignored && ld_acq(&r->h.started) == x->seq) {
      if (g_fault_ignore.load()) {
        x->ignored = true;
      } else {
        x->started = true;
        x->t_started = now_ns();
        const uint64_t us = g_fault_stall_us.load();
        if (us) std::this_thread::sleep_for(std::chrono::microseconds(us));
      }
      p = true;
    }
    // The kernel leaves the record only after `complete`, or on its watchdog
    // (a self-contained kernel leaves when its own entries are done).
    if (!x->completed && !x->aborting && !x->self_contained && ld_acq(&r->h.released) == x->seq) {
      x->aborting = true;
      x->failed = true;
      p = true;
    }
    if (x->ignored || x->aborting) return p;
    // Closed: no more ring entries will ever be appended (every task claimed,
    // or the transfer failed, and no SDMA slot still has a staging step to append).
    if (!x->closed && (x->n_claimed == x->tasks.size() || x->failed) && x->sdma_cu_pending == 0) {
      st_rel(&r->h.cu_total, x->pushed);
      st_rel(&r->h.closed, x->seq);
      close_ring(x);
      x->closed = true;
      p = true;
    }
    // Complete: every micro-task landed -- or, after a failure, everything in
    // flight has drained, so the stream can be released (the error is sticky).
    // The kernel's last wave starts waiting only after every wave has left the
    // ring, i.e. after every appended entry is done; so once the ring is closed,
    // only copy-engine operations can still be outstanding, and `complete` can
    // be published as soon as none is -- without waiting to see the last CU
    // done flags.
    const bool drained = x->failed && x->closed && x->sdma_refs == 0 && x->cu_busy == 0;
    const bool landed = !x->failed && x->closed && sdma_ops_in_flight(x) == 0;
    if (!x->completed && (x->n_done == x->tasks.size() || landed || drained)) {
      st_rel(&r->h.complete, x->seq);
      x->t_complete = now_ns();
      x->completed = true;
      p = true;
    }
    return p;
  }

  void record_trace(const Transfer* x, bool bad) {
    mma_trace_rec_t t{};
    t.seq = x->seq;
    t.dir = x->dir;
    t.kind = static_cast<int32_t>(x->kind);
    t.bytes = x->bytes;
    t.tasks = x->tasks.size();
    t.t_api_ns = x->t_api;
    t.t_submit_ns = x->t_submit;
    t.t_started_ns = x->t_started;
    t.t_first_sdma_ns = x->t_first_sdma;
    t.t_last_task_ns = x->t_last_task;
    t.t_complete_ns = x->t_complete;
    t.t_retire_ns = now_ns();
    for (int i = 0; i < MMA_NUM_PATHS; ++i) t.path_tasks[i] = x->path_tasks[i];
    t.failed = bad ? 1 : 0;
    std::lock_guard<std::mutex> g(g_trace_mu);
    if (g_trace_buf.size() >= kTraceCap) g_trace_buf.pop_front();
    g_trace_buf.push_back(t);
  }

  // Every wave holds at most one claim beyond the last real ticket, so the
  // tickets [pushed, pushed + waves) cover all of them: an end marker in each
  // lets every waiting wave leave on its next poll. The slots are free because
  // push_unit keeps `waves` slots in reserve.
  void close_ring(Transfer* x) {
    Record* r = x->rec;
    for (uint64_t t = x->pushed; t < x->pushed + x->waves; ++t) {
      CuEntry* e = &r->ring[t % kRingSize];
      e->a = 0;
      e->b = 0;
      e->count = 0;
      e->kind_p0 = kEntryEnd;
      const uint64_t tag = make_tag(x->seq, t);
      st_rel(&e->tag0, tag);
      st_rel(&e->tag1, tag);
    }
  }

  // SDMA slots of x whose remaining work includes a copy-engine operation (a
  // slot in kH2DScatter only waits for ring entries, which the kernel finishes).
  int sdma_ops_in_flight(const Transfer* x) const {
    int n = 0;
    for (const auto& s : slots_)
      if (s.x == x && s.state != kFree && s.state != kH2DScatter) ++n;
    return n;
  }

  bool retire_ready(Transfer* x) {
    // A self-contained kernel's done tags are its last accesses to the record.
    if (x->self_contained) return x->n_done == x->tasks.size();
    if (ld_acq(&x->rec->h.released) != x->seq) return false;
    return x->sdma_refs == 0;
  }

  void loop() {
    uint64_t idle_spins = 0, busy_t0 = 0;
    for (;;) {
      if (active_.empty()) {
        if (busy_t0) {
          st_->busy_ns += now_ns() - busy_t0;
          busy_t0 = 0;
        }
        // Back-to-back transfers are common: poll for a while before sleeping,
        // so that a new transfer does not pay a thread wake-up.
        const uint64_t t0 = now_ns();
        while (n_incoming_.load(std::memory_order_acquire) == 0 && !stop_flag_.load(std::memory_order_relaxed) &&
               now_ns() - t0 < kIdleSpinNs)
          cpu_relax();
        std::unique_lock<std::mutex> lk(mu_);
        while (incoming_.empty()) {
          if (stop_) return;
          cv_.wait_for(lk, std::chrono::milliseconds(100));
        }
      }
      if (n_incoming_.load(std::memory_order_acquire) > 0) {
        std::lock_guard<std::mutex> g(mu_);
        while (!incoming_.empty()) {
          active_.push_back(std::move(incoming_.front()));
          incoming_.pop_front();
          n_incoming_.fetch_sub(1, std::memory_order_relaxed);
        }
      }
      if (!busy_t0) busy_t0 = now_ns();
      bool p = false;
      for (auto& up : active_) {
        up->progress = false;
        p |= advance(up.get());
        p |= scan_cu(up.get());
      }
      p |= poll_sdma();
      for (auto& up : active_) p |= pull_cu(up.get());
      p |= pull_sdma();
      for (auto& up : active_) {
        p |= advance(up.get());
        if (up->progress && !up->ignored) st_rel(&up->rec->h.heartbeat, ++up->heartbeat);
      }
      // Retire transfers whose kernel has left the record.
      for (size_t i = 0; i < active_.size();) {
        Transfer* x = active_[i].get();
        if (!retire_ready(x)) {
          ++i;
          continue;
        }
        const bool bad = x->failed || x->ignored || ld_acq(&x->rec->h.status) != 0;
        if (bad) {
          g_sticky.store(1);
          st_->failed += 1;
        }
        st_->transfers += 1;
        if (g_trace.load(std::memory_order_relaxed)) record_trace(x, bad);
        if (x->waiter) {
          std::lock_guard<std::mutex> g(x->waiter->mu);
          x->waiter->done = true;
          x->waiter->failed = bad;
          x->waiter->cv.notify_all();
        }
        {
          std::lock_guard<std::mutex> g(mu_);
          free_recs_.push_back(x->rec_idx);
          --inflight_;
        }
        cv_done_.notify_all();
        active_.erase(active_.begin() + static_cast<long>(i));
        p = true;
      }
      if (p) {
        idle_spins = 0;
      } else if (++idle_spins < 20000) {
        cpu_relax();
      } else {
        std::this_thread::sleep_for(std::chrono::microseconds(20));
      }
    }
  }

  int dir_;
  Config cfg_;
  hsa_agent_t gpu_, cpu_;
  Stats* st_;
  Record* recs_ = nullptr;
  Record* recs_dev_ = nullptr;
  DevState* ds_ = nullptr;
  std::vector<SdmaSlot> slots_;
  std::vector<SdmaPath> paths_;
  uint64_t stage_bytes_ = 0;
  size_t rr_ = 0;
  std::mutex mu_;
  std::condition_variable cv_, cv_done_;
  std::deque<std::unique_ptr<Transfer>> incoming_;
  std::vector<std::unique_ptr<Transfer>> active_;  // engine thread only
  std::deque<uint32_t> free_recs_;
  uint64_t inflight_ = 0;
  bool stop_ = false;
  std::atomic<bool> stop_flag_{false};
  std::atomic<uint64_t> n_incoming_{0};
  static constexpr uint64_t kIdleSpinNs = 2000000;  // 2 ms
  std::thread thread_;
};

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

struct Runtime {
  int dev = 0;
  mma_config_t ucfg{};
  Config cfg{};
  Agents ag;
  uint32_t wallclock_khz = 100000;
  bool hsa_up = false;
  std::unique_ptr<Engine> eng[2];
  std::mutex submit_mu;
  std::atomic<uint64_t> seq{0};
  Stats stats;
};

Runtime* g_rt = nullptr;
std::mutex g_init_mu;

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
  uint64_t id0 = 0, id1 = 0;
  hipDeviceptr_t first = const_cast<void*>(p);
  hipDeviceptr_t last = static_cast<uint8_t*>(const_cast<void*>(p)) + (bytes - 1);
  if (hipPointerGetAttribute(&id0, HIP_POINTER_ATTRIBUTE_BUFFER_ID, first) != hipSuccess ||
      hipPointerGetAttribute(&id1, HIP_POINTER_ATTRIBUTE_BUFFER_ID, last) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return id0 == id1 && id0 != 0;
}

// Pinned, device-mapped host range: returns the device-visible address of p.
mma_status_t host_range(const void* p, uint64_t bytes, uint64_t* dev_addr) {
  hipPointerAttribute_t a{};
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return fail(MMA_ERR_NOT_PINNED, "host pointer %p is not pinned host memory", p);
  }
  if (a.type == hipMemoryTypeDevice) return fail(MMA_ERR_INVALID_ARG, "%p is device memory, host memory expected", p);
  if (a.type != hipMemoryTypeHost || !a.devicePointer)
    return fail(MMA_ERR_NOT_PINNED, "host pointer %p is not pinned, device-mapped host memory", p);
  if (!within_allocation(p, bytes))
    return fail(MMA_ERR_NOT_PINNED, "host range [%p, +%llu) is not inside one pinned allocation", p,
                static_cast<unsigned long long>(bytes));
  *dev_addr = reinterpret_cast<uint64_t>(a.devicePointer);
  return MMA_OK;
}

mma_status_t device_range(const void* p, uint64_t bytes) {
  hipPointerAttribute_t a{};
  if (hipPointerGetAttributes(&a, p) != hipSuccess || a.type != hipMemoryTypeDevice) {
    (void)hipGetLastError();
    return fail(MMA_ERR_INVALID_ARG, "%p is not device memory", p);
  }
  if (a.device != g_rt->dev) return fail(MMA_ERR_INVALID_ARG, "%p belongs to device %d", p, a.device);
  if (!within_allocation(p, bytes))
    return fail(MMA_ERR_INVALID_ARG, "device range [%p, +%llu) is not inside one allocation", p,
                static_cast<unsigned long long>(bytes));
  return MMA_OK;
}

// Workgroups of the dummy-task kernel: one wave per ring entry that can be
// outstanding at once (waves beyond that would only poll host memory, and
// every poll is a PCIe read that competes with the payload).
uint32_t grid_for(const Runtime* rt, Engine* e, uint64_t bytes, uint64_t sub, bool needs_cu, bool staged,
                  bool pool_dev) {
  if (!needs_cu) return 1;
  if (pool_dev) {  // HBM gather/scatter: as many waves as there are micro-tasks, up to the limit
    const uint64_t tasks = (bytes + rt->cfg.chunk - 1) / rt->cfg.chunk;
    return static_cast<uint32_t>(std::max<uint64_t>(1, std::min<uint64_t>((tasks + 3) / 4, kMaxWorkgroups)));
  }
  const Config& c = rt->cfg;
  const uint64_t total = (bytes + sub - 1) / sub;
  const uint64_t per_task = (c.chunk + sub - 1) / sub;
  uint64_t inflight = e->cu_enabled() ? c.cu_depth * per_task : 0;
  if (staged) inflight += static_cast<uint64_t>(__builtin_popcount(e->sdma_mask())) * c.depth * per_task;
  uint64_t g = (std::max<uint64_t>(1, std::min(total, inflight)) + kWavesPerWG - 1) / kWavesPerWG;
  g = std::max<uint64_t>(1, std::min<uint64_t>(g, c.cu_wgs));
  return static_cast<uint32_t>(g);
}

// Hand a planned transfer to its engine and enqueue the dummy task on the stream.
struct KvGeom {
  uint64_t piece = 0, kstride = 0;
  uint32_t layers = 0;
  uint64_t layer_ptr[kMaxLayers];
};

mma_status_t submit(std::unique_ptr<Transfer> x, uint64_t payload_bytes, void* stream, const KvGeom* kv) {
  Runtime* rt = g_rt;
  Engine* e = rt->eng[x->dir].get();
  x->claimed.assign(x->tasks.size(), 0);
  x->left.assign(x->tasks.size(), 0);
  std::lock_guard<std::mutex> g(rt->submit_mu);
  if (!e->acquire_record(x.get(), 60000)) return fail(MMA_ERR_TIMEOUT, "no free transfer record for 60 s");
  x->seq = ++rt->seq;
  x->t_submit = now_ns();
  x->bytes = payload_bytes;
  Record* r = x->rec;
  r->h.seq = x->seq;
  r->h.status = 0;
  __atomic_thread_fence(__ATOMIC_RELEASE);
  if (rt->cfg.static_split && e->has_sdma() && x->sdma_ok) {
    for (size_t i = 0; i < x->tasks.size(); ++i) {
      uint32_t& f = x->tasks[i].flags;
      if (f & kPlanCuOnly) continue;
      f |= static_cu_task(i, rt->cfg.static_cu_percent) ? kPlanCuOnly : kPlanSdmaOnly;
    }
  }
  const bool staged = x->kind != Kind::kLinear && e->has_sdma() && x->sdma_ok;
  const bool needs_cu = e->cu_enabled() || staged ||
                        std::any_of(x->tasks.begin(), x->tasks.end(),
                                    [](const Task& t) { return (t.flags & kPlanCuOnly) != 0; });
  // CU ring entries of a linear transfer are cu_sub_bytes. A transfer that can
  // fit the launch's prefilled entries is cut finer (16 KiB steps, one wave
  // register batch), so that more waves share it and it costs about one PCIe
  // round trip.
  x->sub = rt->cfg.sub;
  if (!kv && payload_bytes <= kPrefill * rt->cfg.sub) {
    const uint64_t per = (payload_bytes + kPrefill - 1) / kPrefill;
    x->sub = std::min<uint64_t>(rt->cfg.sub, std::max<uint64_t>(kSmallSub, (per + kSmallSub - 1) / kSmallSub * kSmallSub));
  }
  uint32_t grid = grid_for(rt, e, payload_bytes, x->sub, needs_cu || x->pool_dev, staged, x->pool_dev);
  x->waves = grid * kWavesPerWG;
  e->prefill(x.get());
  const uint32_t n_pre = kv ? 0u : static_cast<uint32_t>(std::min<uint64_t>(x->pushed, kPrefill));
  // Everything fits the launch: all tasks were claimed by the CU prefill (so no
  // copy engine can take part) and all their entries are in the kernel args.
  // One wave per entry; the engine treats the transfer as started.
  x->self_contained = !kv && x->n_claimed == x->tasks.size() && x->pushed == n_pre;
  if (x->self_contained) {
    grid = (n_pre + kWavesPerWG - 1) / kWavesPerWG;
    x->waves = grid * kWavesPerWG;
    x->started = true;
    x->t_started = x->t_submit;
  }
  if (tl_waiter) {
    x->waiter = tl_waiter;
    tl_waiter->submitted = true;
  }
  static thread_local KernelArgs a;
  memset(&a, 0, offsetof(KernelArgs, layer_ptr));
  a.n_pre = n_pre;
  a.self_contained = x->self_contained ? 1u : 0u;
  for (uint32_t t = 0; t < n_pre; ++t) {
    const CuEntry& en = r->ring[t];
    a.pre[t][0] = en.a;
    a.pre[t][1] = en.b;
    a.pre[t][2] = static_cast<uint64_t>(en.count) | (static_cast<uint64_t>(en.kind_p0) << 32);
  }
  if (kv) {
    a.kv_piece_bytes = kv->piece;
    a.kv_kstride = kv->kstride;
    a.kv_layers = kv->layers;
    memcpy(a.layer_ptr, kv->layer_ptr, sizeof(uint64_t) * kv->layers);
  }
  a.rec = e->rec_dev(x->rec_idx);
  a.ds = e->ds(x->rec_idx);
  a.seq = x->seq;
  a.watchdog_ticks = static_cast<uint64_t>(rt->cfg.watchdog_ms) * rt->wallclock_khz;
  a.total_waves = grid * kWavesPerWG;
  a.release_each = x->dir == MMA_D2H ? 1u : 0u;
  DeviceGuard dg(rt->dev);
  const hipError_t err = launch_transfer(a, grid, static_cast<hipStream_t>(stream));
  if (err != hipSuccess) {
    e->release_record_unused(x.get());
    return fail(MMA_ERR_HIP, "dummy-task kernel launch failed: %s", hipGetErrorString(err));
  }
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
  if (use_env) {
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
  }
  *c = d;
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

mma_status_t mma_init(int hip_device, const mma_config_t* user_cfg) {
  std::lock_guard<std::mutex> g(g_init_mu);
  if (g_rt) return fail(MMA_ERR_ALREADY_INITIALIZED, "already initialised");
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || hip_device < 0 || hip_device >= ndev) {
    (void)hipGetLastError();
    return fail(MMA_ERR_INVALID_ARG, "invalid HIP device %d (%d devices)", hip_device, ndev);
  }
  mma_config_t c;
  if (user_cfg) {
    mma_config_t d;
    fill_config(&d, false);
    c = *user_cfg;
    if (!c.chunk_bytes) c.chunk_bytes = d.chunk_bytes;
    if (!c.small_bytes) c.small_bytes = d.small_bytes;
    if (!c.queue_depth) c.queue_depth = d.queue_depth;
    if (!c.cu_queue_depth) c.cu_queue_depth = d.cu_queue_depth;
    if (!c.cu_workgroups) c.cu_workgroups = d.cu_workgroups;
    if (!c.cu_sub_bytes) c.cu_sub_bytes = d.cu_sub_bytes;
    if (!c.watchdog_ms) c.watchdog_ms = d.watchdog_ms;
  } else {
    fill_config(&c, true);
  }
  if (!c.fallback_bytes) c.fallback_bytes = 2 * c.chunk_bytes;
  // A micro-task's ring entries must fit the ring next to the end-marker
  // reserve of one slot per wave.
  if (c.cu_sub_bytes % 16 || c.cu_sub_bytes < 256 || c.chunk_bytes % 16 || c.queue_depth > 16 ||
      c.cu_workgroups > kMaxWorkgroups || c.cu_queue_depth > 64 ||
      (c.chunk_bytes + c.cu_sub_bytes - 1) / c.cu_sub_bytes > kRingSize / 2)
    return fail(MMA_ERR_INVALID_ARG, "invalid configuration");

  std::unique_ptr<Runtime> rt(new Runtime());
  rt->dev = hip_device;
  DeviceGuard dg(hip_device);
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, hip_device) != hipSuccess) return fail(MMA_ERR_HIP, "hipGetDeviceProperties");
  int wclk = 0;
  if (hipDeviceGetAttribute(&wclk, hipDeviceAttributeWallClockRate, hip_device) == hipSuccess && wclk > 0)
    rt->wallclock_khz = static_cast<uint32_t>(wclk);
  if (hsa_init() != HSA_STATUS_SUCCESS) return fail(MMA_ERR_HSA, "hsa_init failed");
  rt->hsa_up = true;
  rt->ag.want_bdf = static_cast<uint32_t>((prop.pciBusID << 8) | (prop.pciDeviceID << 3));
  rt->ag.want_domain = static_cast<uint32_t>(prop.pciDomainID);
  hsa_iterate_agents(agent_cb, &rt->ag);
  if (!rt->ag.have_gpu || !rt->ag.have_cpu) {
    hsa_shut_down();
    return fail(MMA_ERR_HSA, "no ROCr agent for HIP device %d", hip_device);
  }
  uint32_t avail[2] = {0, 0}, nsdma = 0;
  hsa_amd_memory_copy_engine_status(rt->ag.gpu, rt->ag.cpu, &avail[MMA_H2D]);
  hsa_amd_memory_copy_engine_status(rt->ag.cpu, rt->ag.gpu, &avail[MMA_D2H]);
  hsa_agent_get_info(rt->ag.gpu, static_cast<hsa_agent_info_t>(HSA_AMD_AGENT_INFO_NUM_SDMA_ENG), &nsdma);
  const uint32_t host_facing = nsdma >= 16 ? 0xFFFFu : ((1u << nsdma) - 1u);
  uint32_t mask[2] = {c.path_mask_h2d, c.path_mask_d2h};
  for (int d = 0; d < 2; ++d) {
    if (!mask[d]) mask[d] = MMA_PATH_CU | (avail[d] & host_facing);
    mask[d] = (mask[d] & MMA_PATH_CU) | (mask[d] & avail[d] & 0xFFFFu);
    if (!(mask[d] & 0xFFFFu)) mask[d] |= MMA_PATH_CU;  // some path must carry the work
  }
  c.path_mask_h2d = mask[0];
  c.path_mask_d2h = mask[1];
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
  k.cu_wgs = c.cu_workgroups;
  k.watchdog_ms = c.watchdog_ms;
  k.mask[0] = mask[0];
  k.mask[1] = mask[1];
  if (c.static_cu_percent > 100) return fail(MMA_ERR_INVALID_ARG, "static_cu_percent > 100");
  k.static_split = c.static_split;
  k.static_cu_percent = c.static_cu_percent;
  k.merge = c.sdma_merge_tasks ? c.sdma_merge_tasks
                              : static_cast<uint32_t>(std::max<uint64_t>(1, 8 * MiB / c.chunk_bytes));

  // SDMA staging for the KV kinds: one chunk per SDMA slot, in uncached device
  // memory (coherent between the copy engines and every XCD's L2 without
  // cache maintenance). Kept for the process lifetime and reused.
  const uint64_t stage_bytes = (std::max<uint64_t>(k.chunk, 2 * MiB) + 4095) & ~4095ull;
  for (int d = 0; d < 2; ++d) {
    const uint32_t n = static_cast<uint32_t>(__builtin_popcount(mask[d] & 0xFFFFu));
    const uint64_t need = n * k.depth * stage_bytes;
    StagingCache& sc = g_staging[d];
    if (need && (sc.dev != hip_device || sc.bytes < need)) {
      void* p = nullptr;
      if (hipExtMallocWithFlags(&p, need, hipDeviceMallocUncached) != hipSuccess) {
        (void)hipGetLastError();
        hsa_shut_down();
        return fail(MMA_ERR_HIP, "staging allocation of %llu bytes failed", static_cast<unsigned long long>(need));
      }
      sc.dev = hip_device;
      sc.base = p;
      sc.bytes = need;
    }
  }
  for (int d = 0; d < 2; ++d) {
    rt->eng[d].reset(new Engine(d, k, rt->ag.gpu, rt->ag.cpu, &rt->stats));
    mma_status_t s = rt->eng[d]->init(mask[d] & 0xFFFFu, stage_bytes, (mask[d] & 0xFFFFu) ? g_staging[d].base : nullptr);
    if (s != MMA_OK) {
      rt->eng[0].reset();
      rt->eng[1].reset();
      hsa_shut_down();
      return s;
    }
    set_affinity_local(rt->eng[d]->native_handle(), hip_device);
  }
  if (env_u64("MMA_TRACE", 0)) g_trace = 1;
  g_rt = rt.release();
  return MMA_OK;
}

mma_status_t mma_finalize(void) {
  std::lock_guard<std::mutex> g(g_init_mu);
  if (!g_rt) return fail(MMA_ERR_NOT_INITIALIZED, "not initialised");
  bool drained = true;
  for (auto& e : g_rt->eng) drained = e->wait_idle(30000) && drained;
  if (!drained) return fail(MMA_ERR_TIMEOUT, "in-flight transfers did not drain");
  {
    DeviceGuard dg(g_rt->dev);
    for (auto& e : g_rt->eng) e.reset();
  }
  if (g_rt->hsa_up) hsa_shut_down();
  delete g_rt;
  g_rt = nullptr;
  return MMA_OK;
}

mma_status_t mma_get_config(mma_config_t* out) {
  if (!out) return fail(MMA_ERR_INVALID_ARG, "NULL config");
  if (!g_rt) return fail(MMA_ERR_NOT_INITIALIZED, "not initialised");
  *out = g_rt->ucfg;
  return MMA_OK;
}

mma_status_t mma_synchronize(uint32_t timeout_ms) {
  if (!g_rt) return fail(MMA_ERR_NOT_INITIALIZED, "not initialised");
  for (auto& e : g_rt->eng)
    if (!e->wait_idle(timeout_ms)) return fail(MMA_ERR_TIMEOUT, "transfers still in flight");
  return g_sticky.load() ? fail(MMA_ERR_TRANSFER_FAILED, "a transfer failed") : MMA_OK;
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

mma_status_t mma_memcpy(void* dst, const void* src, uint64_t bytes, int32_t dir) {
  std::shared_ptr<Waiter> w = std::make_shared<Waiter>();
  tl_waiter = w;
  mma_status_t s = mma_memcpy_async(dst, src, bytes, dir, nullptr);
  tl_waiter.reset();
  if (s) return s;
  if (!w->submitted) return MMA_OK;  // nothing to move
  {
    DeviceGuard dg(g_rt->dev);
    const hipError_t e = hipStreamSynchronize(nullptr);
    if (e != hipSuccess) return fail(MMA_ERR_HIP, "hipStreamSynchronize: %s", hipGetErrorString(e));
  }
  // The stream has passed the dummy task; the engine retires the transfer
  // right after, which is when its outcome is final.
  std::unique_lock<std::mutex> lk(w->mu);
  const uint64_t ms = static_cast<uint64_t>(g_rt->cfg.watchdog_ms) + 10000;
  if (!w->cv.wait_for(lk, std::chrono::milliseconds(ms), [&] { return w->done; }))
    return fail(MMA_ERR_TIMEOUT, "copy not retired");
  return w->failed ? fail(MMA_ERR_TRANSFER_FAILED, "the copy failed") : MMA_OK;
}

mma_status_t mma_weights_load(const mma_copy_desc_t* list, uint64_t n, int32_t dir, void* stream) {
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
  std::vector<PlanItem> plan;
  plan_list(sizes.data(), n, rt->cfg.chunk, rt->cfg.fallback, rt->cfg.small, plan);
  std::unique_ptr<Transfer> x(new Transfer());
  x->dir = dir;
  x->t_api = t_api;
  x->kind = Kind::kLinear;
  x->tasks.reserve(plan.size());
  for (const PlanItem& p : plan) {
    const mma_copy_desc_t& d = list[p.item];
    Task t{};
    t.src_dma = reinterpret_cast<uint64_t>(d.src) + p.offset;
    t.dst_dma = reinterpret_cast<uint64_t>(d.dst) + p.offset;
    t.src_cu = src_cu[p.item] + p.offset;
    t.dst_cu = dst_cu[p.item] + p.offset;
    t.bytes = p.bytes;
    t.flags = p.flags;
    x->tasks.push_back(t);
  }
  return submit(std::move(x), total, stream, nullptr);
}

static mma_status_t kv_common(const mma_kv_layout_t* lay, const void* host_pool, const void* const* layers,
                              const int32_t* host_slots, const int32_t* gpu_blocks, uint64_t n, int dir,
                              void* stream) {
  const uint64_t t_api = now_ns();
  mma_status_t s = check_ready();
  if (s) return s;
  if (!n) return MMA_OK;
  if (!lay || !host_pool || !layers || !host_slots || !gpu_blocks)
    return fail(MMA_ERR_INVALID_ARG, "NULL argument");
  if (!lay->num_layers || lay->num_layers > kMaxLayers || !lay->block_tokens || !lay->kv_heads || !lay->head_dim ||
      !lay->elem_bytes || !lay->gpu_num_blocks || !lay->host_num_slots)
    return fail(MMA_ERR_INVALID_ARG, "invalid KV layout");
  const uint64_t piece = static_cast<uint64_t>(lay->block_tokens) * lay->kv_heads * lay->head_dim * lay->elem_bytes;
  if (piece > (1ull << 32)) return fail(MMA_ERR_INVALID_ARG, "KV piece too large");
  const uint32_t ppb = 2 * lay->num_layers;
  const uint64_t slot_bytes = piece * ppb;
  const uint64_t pool_bytes = slot_bytes * lay->host_num_slots;
  const uint64_t layer_bytes = 2 * piece * lay->gpu_num_blocks;
  bool ok = dir == MMA_H2D ? tables_valid(host_slots, lay->host_num_slots, gpu_blocks, lay->gpu_num_blocks, n)
                           : tables_valid(gpu_blocks, lay->gpu_num_blocks, host_slots, lay->host_num_slots, n);
  if (!ok) return fail(MMA_ERR_INVALID_ARG, "block table entry out of range or duplicate destination");
  Runtime* rt = g_rt;
  DeviceGuard dg(rt->dev);
  // The pool is pinned host memory, or device memory of this GPU (a KV tier
  // in HBM): then the transfer is an HBM gather/scatter carried by the CU path.
  uint64_t pool_cu = 0;
  bool pool_dev = false;
  if ((s = host_range(host_pool, pool_bytes, &pool_cu))) {
    const std::string host_err = t_err;
    if (s != MMA_ERR_INVALID_ARG || device_range(host_pool, pool_bytes) != MMA_OK) {
      t_err = host_err;
      return s;
    }
    pool_dev = true;
    pool_cu = reinterpret_cast<uint64_t>(host_pool);
  }
  KvGeom kv;
  kv.layers = lay->num_layers;
  kv.piece = piece;
  kv.kstride = piece * lay->gpu_num_blocks;
  for (uint32_t l = 0; l < lay->num_layers; ++l) {
    if (!layers[l]) return fail(MMA_ERR_INVALID_ARG, "NULL layer pointer %u", l);
    if ((s = device_range(layers[l], layer_bytes))) return s;
    kv.layer_ptr[l] = reinterpret_cast<uint64_t>(layers[l]);
  }
  std::vector<PlanItem> plan;
  plan_kv(n, ppb, piece, rt->cfg.chunk, plan);
  std::unique_ptr<Transfer> x(new Transfer());
  x->dir = dir;
  x->t_api = t_api;
  x->kind = dir == MMA_H2D ? Kind::kKvFetch : Kind::kKvOffload;
  x->piece = piece;
  Engine* e = rt->eng[dir].get();
  const uint64_t per_task = std::max<uint64_t>(rt->cfg.chunk / piece, 1) * piece;
  x->pool_dev = pool_dev;
  x->sdma_ok = per_task <= e->stage_bytes() && !pool_dev;
  x->tasks.reserve(plan.size());
  const uint64_t host = reinterpret_cast<uint64_t>(host_pool);
  for (const PlanItem& p : plan) {
    Task t{};
    const uint64_t off = static_cast<uint64_t>(host_slots[p.item]) * slot_bytes + p.offset * piece;
    t.host_dma = host + off;
    t.host_cu = pool_cu + off;
    t.blk = static_cast<uint64_t>(gpu_blocks[p.item]);
    t.p0 = static_cast<uint32_t>(p.offset);
    t.bytes = p.bytes;
    t.flags = x->sdma_ok ? 0u : kPlanCuOnly;
    x->tasks.push_back(t);
  }
  return submit(std::move(x), n * slot_bytes, stream, &kv);
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

mma_status_t mma_get_stats(mma_stats_t* out) {
  if (!out) return fail(MMA_ERR_INVALID_ARG, "NULL out");
  if (!g_rt) return fail(MMA_ERR_NOT_INITIALIZED, "not initialised");
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
    default: return "MMA_ERR_UNKNOWN";
  }
}

const char* mma_last_error(void) { return t_err.c_str(); }

mma_status_t mma_clear_error(void) {
  g_sticky.store(0);
  t_err.clear();
  return MMA_OK;
}

mma_status_t mma_trace_enable(int32_t on) {
  std::lock_guard<std::mutex> g(g_trace_mu);
  if (on && !g_trace.load()) g_trace_buf.clear();
  g_trace = on ? 1 : 0;
  return MMA_OK;
}

mma_status_t mma_trace_read(mma_trace_rec_t* out, uint64_t cap, uint64_t* n_out) {
  if (!n_out || (cap && !out)) return fail(MMA_ERR_INVALID_ARG, "NULL argument");
  std::lock_guard<std::mutex> g(g_trace_mu);
  const uint64_t n = std::min<uint64_t>(cap, g_trace_buf.size());
  for (uint64_t i = 0; i < n; ++i) out[i] = g_trace_buf[i];
  g_trace_buf.erase(g_trace_buf.begin(), g_trace_buf.begin() + static_cast<long>(n));
  *n_out = n;
  return MMA_OK;
}

mma_status_t mma_test_set_fault(int32_t kind, uint64_t value) {
  switch (kind) {
    case MMA_FAULT_ENGINE_STALL_US: g_fault_stall_us = value; return MMA_OK;
    case MMA_FAULT_SDMA_SUBMIT_FAIL: g_fault_submit_fail = value; return MMA_OK;
    case MMA_FAULT_ENGINE_IGNORE: g_fault_ignore = value; return MMA_OK;
    default: return fail(MMA_ERR_INVALID_ARG, "unknown fault kind %d", kind);
  }
}

}  // extern "C"
