// Host engine of the multipath copy path, independent of the GPU runtime: the
// transfer bookkeeping, the per-direction engine thread (Section 4: separate
// H2D and D2H engine instances) with its path selector, copy-engine slots and
// CU-ring protocol, and the micro-task builders. Everything that touches the
// GPU goes through Backend: ROCr/HIP in mma_runtime.cpp, host threads in the
// CPU engine test.
//
// Roles, mapped to the paper's components (Section 3, Figure "Overview"):
//   Task Manager   -> make_*_transfer (plans from mma_plan.cpp) + per-task
//                     completion accounting (Engine::task_done).
//   Path Selector  -> Engine::pull_cu / Engine::pull_sdma: every path pulls the
//                     next micro-task only while its outstanding queue has
//                     room (backpressure).
//   Task Launcher  -> Backend::copy (SDMA) and ring entries consumed by the
//                     dummy-task kernel (CU path).
//   Sync Engine    -> the record's started/complete words (Engine::advance).
// Under device control (Engine::prepare_device) the submitting thread plans
// the whole transfer and the kernel tracks its completion: no engine-thread
// work per transfer.
#ifndef MMA_ENGINE_H_
#define MMA_ENGINE_H_

#include <pthread.h>
#include <sys/prctl.h>
#include <time.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdarg>
#include <cstddef>
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

// ------------------------------------------------------------------ utilities
inline thread_local std::string t_err;  // message of the calling thread's last error

inline mma_status_t fail(mma_status_t s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  t_err = buf;
  return s;
}

inline uint64_t now_ns() {
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

inline uint64_t env_u64(const char* name, uint64_t dflt) {
  const char* v = getenv(name);
  if (!v || !*v) return dflt;
  return strtoull(v, nullptr, 0);
}

constexpr uint64_t KiB = 1024, MiB = 1024 * 1024;
constexpr uint64_t kSmallSub = 16 * KiB;  // one wave register batch
// CU entry size behind the default size limit of transfers taken whole by the
// CU path: kPrefill entries of this size travel in the launch arguments (24 MiB).
constexpr uint64_t kWholeMaxSub = 512 * KiB;
// Device control: default CU-path share of a linear transfer's bytes when the
// copy engines take part (the rest is split between the engines). Measured on
// 1 GiB copies, 40% to 70% land within 0.2% of each other; 40% was best in
// both directions.
constexpr uint32_t kDeviceCuPercent = 40;
// Device control: a copy or tensor list with more micro-tasks than a ring is
// planned again at twice the chunk size, up to this chunk (a CU entry's byte
// count is 32 bits).
constexpr uint64_t kDeviceMaxChunk = 1ull << 30;

// ------------------------------------------------------------------ transfer
enum class Kind : uint8_t { kLinear, kKvFetch, kKvOffload };

// Completion slot of one synchronous call (mma_memcpy): set by the engine
// thread when it retires the transfer.
struct Waiter {
  std::mutex mu;
  std::condition_variable cv;
  bool submitted = false, done = false, failed = false;
};
inline thread_local std::shared_ptr<Waiter> tl_waiter;

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
  Record* rec = nullptr;      // host address of the shared record; null for a light slot
  int32_t light = -1;         // light slot (a whole self-contained transfer), or -1
  CuEntry* ring = nullptr;    // where the engine writes ring entries (the record's, or a scratch ring)
  uint64_t* done_host = nullptr;  // done tags the kernel writes
  std::vector<Task> tasks;
  std::vector<uint8_t> claimed;
  std::vector<uint32_t> left;  // CU entries outstanding per CU-path task
  size_t cur_cu = 0, cur_sdma = 0, n_claimed = 0, n_done = 0;
  size_t cu_only_left = 0, cur_cu_only = 0;  // unclaimed CU-only micro-tasks; scan cursor while the CU path pauses
  uint64_t piece = 0;
  bool sdma_ok = true;         // SDMA may carry this transfer's tasks
  // CU ring bookkeeping
  uint64_t pushed = 0, done_upto = 0;
  uint32_t waves = 0;          // waves of the dummy-task kernel
  bool pool_dev = false;       // KV pool in device memory: HBM gather/scatter, one entry per task
  // HBM pool launch: the transfer is one launch of the pool kernel, which reads
  // the block table (pool slot | GPU block << 32 per block) from the engine's
  // table arena, segments [tab_seg, tab_seg + tab_nseg).
  bool pool_launch = false;
  uint64_t pool_base = 0;
  std::vector<uint64_t> pool_pairs;
  int32_t tab_seg = -1;
  uint32_t tab_nseg = 0;
  bool self_contained = false; // whole transfer in the kernel args; the kernel does not wait on the host
  bool whole = false;          // the CU path claims every micro-task at prefill
  // Submitted on a stream with nothing pending: the engine may start the copy
  // engines at once, without waiting for the kernel's start signal.
  bool early = false;
  // Set by the submitting thread when the dummy-task launch of an early
  // transfer failed: no kernel will ever run for it.
  std::atomic<bool> unlaunched{false};
  uint64_t sub = 0;            // bytes per CU ring entry of a linear transfer
  uint64_t kv_per = 0;         // pieces per CU ring entry of a KV transfer (0: the engine thread's rule)
  // Device control: planned in full at submission (prepare_device), retired by reap.
  uint32_t dev_cmds = 0;           // copy-engine commands counted by the record's device signal
  bool dev_hold = false;           // test fault: the signal counts one command too many until reaped
  std::vector<uint8_t> dev_path;   // path (stats index) that carries each micro-task
  std::shared_ptr<Waiter> waiter;  // set for synchronous calls
  // Per ring slot (kRingSize of them for a record, kPrefill for a light slot), set
  // when an entry is appended (left uninitialised until then):
  std::unique_ptr<int32_t[]> owner;  // >= 0: CU-path task; < 0: -(1 + SDMA slot id)
  std::unique_ptr<uint8_t[]> tdone;  // its done tag has been seen
  uint32_t cu_busy = 0;
  uint64_t cu_entries = 0;     // ring entries of CU-path micro-tasks appended and not seen done
  bool cu_full = false;
  int sdma_cu_pending = 0;     // SDMA slots that may still append ring entries (a staging step, or a
                               // re-route of their micro-tasks to the CU path)
  int sdma_refs = 0;           // SDMA slots referencing this transfer
  uint64_t heartbeat = 0;
  uint64_t bytes = 0;          // payload bytes
  uint64_t done_bytes = 0;     // payload bytes of the micro-tasks landed so far (engine thread)
  // trace timestamps (CLOCK_MONOTONIC ns)
  uint64_t t_api = 0, t_submit = 0, t_started = 0, t_first_sdma = 0, t_last_task = 0, t_complete = 0;
  uint64_t t_released = 0;     // when the kernel was seen to release the record with tags still missing
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
  uint64_t sig = 0;       // copy-engine completion signal (Backend handle)
  int state = kFree;
  Transfer* x = nullptr;
  size_t task = 0, task_end = 0;  // micro-tasks [task, task_end) carried by this slot's command
  uint64_t count = 0;     // their total: bytes (linear) or pieces (KV, one block's run)
  uint32_t left = 0;      // ring entries outstanding
  uint64_t staging = 0;   // device address of this slot's staging buffer
  int path = 0;
  uint64_t t_submit = 0;  // current copy-engine command: submission time and size
  uint64_t op_bytes = 0;
  uint64_t ahead = 0;     // the other direction's bytes on the same engine at submission: the engine
                          // runs one in-order queue, so they may all run before this command
};

struct SdmaPath {
  int engine = 0;
  std::vector<int> slots;  // slot ids
  int busy = 0;
  bool full = false;
  bool congested = false;  // a command is long overdue: pull nothing more until the engine drains
  uint64_t t_head = 0;     // when the path's oldest command in flight reached the head of its queue
  double ns_per_byte = 0;  // measured time per byte of its commands (moving average; 0: none yet)
};

struct Config {
  uint64_t chunk, fallback, small, sub;
  uint32_t depth, cu_depth, backoff, cu_wgs, watchdog_ms;
  uint32_t cu_backoff;  // the CU path's back-off depth (0: cu_depth, no extra back-off); `backoff` is the engines'
  uint32_t mask[2];
  uint32_t static_split, static_cu_percent;
  uint32_t merge;       // max micro-tasks per copy-engine command
  uint64_t whole[2];    // per direction: transfers up to this size may be taken whole by the CU path (0: never)
  uint32_t device;      // 1: device control (no engine thread in the loop)
  uint32_t device_cu_percent;  // device control: the CU path's share of a linear transfer's bytes
  uint32_t overdue_gbs;        // link rate the overdue rule assumes, GB/s (0: 50)
  uint32_t duplex[2];          // per direction: the paths used while the other direction moves (see set_peer)
  uint64_t nap_ns;             // longest sleep of the engine thread between rounds (see nap); 0: poll
  uint64_t duplex_hold_ns;     // a direction counts as moving this long after it was last seen moving
                               // (0: kDuplexHoldNs)
};

struct Stats {
  std::atomic<uint64_t> transfers{0}, failed{0}, staging_bytes{0}, submit_failures{0}, busy_ns{0};
  std::atomic<uint64_t> foreign_skips{0}, congestion_backoffs{0}, sdma_commands{0}, pool_launches{0}, naps{0};
  std::atomic<uint64_t> path_bytes[MMA_NUM_PATHS], path_tasks[MMA_NUM_PATHS];
  Stats() {
    for (auto& v : path_bytes) v = 0;
    for (auto& v : path_tasks) v = 0;
  }
  void reset() {
    transfers = failed = staging_bytes = submit_failures = busy_ns = foreign_skips = congestion_backoffs = 0;
    sdma_commands = pool_launches = naps = 0;
    for (auto& v : path_bytes) v = 0;
    for (auto& v : path_tasks) v = 0;
  }
};

inline std::atomic<int> g_sticky{0};

// Per-transfer trace records (MMA_TRACE=1 or mma_trace_enable): a bounded ring.
inline std::atomic<int> g_trace{0};
inline std::mutex g_trace_mu;
inline std::deque<mma_trace_rec_t> g_trace_buf;
constexpr size_t kTraceCap = 65536;
inline std::atomic<uint64_t> g_fault_stall_us{0}, g_fault_submit_fail{0}, g_fault_ignore{0};
inline std::atomic<uint64_t> g_fault_signal_hold{0}, g_fault_pool_no_table{0};

// What the engine needs from the GPU side. The product backend is ROCr/HIP
// (mma_runtime.cpp); a CPU test backend emulates it with host threads.
struct Backend {
  virtual ~Backend() = default;
  // Coherent host memory that the device reads and writes (the records);
  // *dev receives the device's address for it.
  virtual mma_status_t alloc_records(uint64_t bytes, void** host, void** dev) = 0;
  virtual void free_records(void* host) = 0;
  // Zero-filled device memory (per-record device state).
  virtual mma_status_t alloc_device_state(uint64_t bytes, void** dev) = 0;
  virtual void free_device_state(void* dev) = 0;
  virtual mma_status_t alloc_host_scratch(uint64_t bytes, void** host) = 0;
  virtual void free_host_scratch(void* host) = 0;
  // Completion signals of copy-engine commands: set to 1 before a command,
  // 0 when it has landed, negative if it failed.
  virtual bool signal_create(uint64_t* sig) = 0;
  virtual void signal_destroy(uint64_t sig) = 0;
  virtual void signal_store(uint64_t sig, int64_t value) = 0;
  virtual int64_t signal_load(uint64_t sig) = 0;
  // One command on copy engine `engine`; false if it was not accepted. The
  // command decrements `sig` by one when it has landed.
  virtual bool copy(int engine, void* dst, bool dst_on_device, const void* src, bool src_on_device,
                    uint64_t bytes, uint64_t sig) = 0;
  // Device control: a completion signal that kernels poll; *value receives the
  // device-visible address of its 64-bit value. false: not available.
  virtual bool signal_create_polled(uint64_t* sig, const int64_t** value) = 0;
  // Atomically subtracts v from the signal's value.
  virtual void signal_sub(uint64_t sig, int64_t v) = 0;
  // Bit e set: copy engine e has no command queued for direction `dir`.
  virtual uint32_t engines_idle(int dir) = 0;
};

// KV geometry handed to the kernel: piece size, K-to-V stride in a layer
// tensor, and the layer tensors' addresses.
struct KvGeom {
  uint64_t piece = 0, kstride = 0;
  uint32_t layers = 0;
  uint32_t layout = kKvLayoutPiece;
  uint32_t tokens = 0, heads = 0, row_bytes = 0, elem = 0, lds_wave = 0;  // x-packed layout
  uint64_t layer_ptr[kMaxLayers];
};

class Engine {
 public:
  Engine(int dir, const Config& cfg, Backend* be, Stats* st) : dir_(dir), cfg_(cfg), be_(be), st_(st) {}
  ~Engine() { shutdown(); }

  mma_status_t init(uint32_t sdma_mask, uint64_t stage_bytes, void* staging_base) {
    void *h = nullptr, *d = nullptr;
    mma_status_t rc = be_->alloc_records(sizeof(Record) * kRecords, &h, &d);
    if (rc != MMA_OK) return rc;
    recs_ = static_cast<Record*>(h);
    recs_dev_ = static_cast<Record*>(d);
    memset(recs_, 0, sizeof(Record) * kRecords);
    if ((rc = be_->alloc_device_state(sizeof(DevState) * kRecords, &d)) != MMA_OK) return rc;
    ds_ = static_cast<DevState*>(d);
    for (uint32_t i = 0; i < kRecords; ++i) free_recs_.push_back(i);
    if ((rc = be_->alloc_records(sizeof(uint64_t) * kPrefill * kLightSlots, &h, &d)) != MMA_OK) return rc;
    light_ = static_cast<uint64_t*>(h);
    light_dev_ = static_cast<uint64_t*>(d);
    memset(light_, 0, sizeof(uint64_t) * kPrefill * kLightSlots);
    for (uint32_t i = 0; i < kLightSlots; ++i) free_light_.push_back(i);
    light_ring_.reset(new CuEntry[kPrefill + kRingSize]);
    if ((rc = be_->alloc_records(sizeof(uint64_t) * kPoolTabEntries, &h, &d)) != MMA_OK) return rc;
    pool_tab_ = static_cast<uint64_t*>(h);
    pool_tab_dev_ = static_cast<uint64_t*>(d);
    if ((rc = be_->alloc_device_state(sizeof(uint32_t) * kLightSlots, &d)) != MMA_OK) return rc;
    pool_ctr_ = static_cast<uint32_t*>(d);
    seg_used_.assign(kPoolTabEntries / kPoolTabSeg, 0);
    stage_bytes_ = stage_bytes;
    uint8_t* stage = static_cast<uint8_t*>(staging_base);
    for (int eng = 0; eng < MMA_MAX_SDMA; ++eng) {
      if (!(sdma_mask & (1u << eng))) continue;
      SdmaPath p;
      p.engine = eng;
      for (uint32_t d = 0; d < cfg_.depth; ++d) {
        SdmaSlot s;
        if (!be_->signal_create(&s.sig)) return fail(MMA_ERR_HSA, "copy-engine signal creation failed");
        s.staging = stage ? reinterpret_cast<uint64_t>(stage) : 0;
        if (stage) stage += stage_bytes;
        s.path = static_cast<int>(paths_.size());
        p.slots.push_back(static_cast<int>(slots_.size()));
        slots_.push_back(s);
      }
      paths_.push_back(p);
    }
    // Device control: one polled completion signal per record for the copy
    // engines' share. Without them the CU path carries device-controlled
    // transfers alone.
    if (cfg_.device && !paths_.empty()) {
      for (uint32_t i = 0; i < kRecords; ++i) {
        uint64_t sig = 0;
        const int64_t* val = nullptr;
        if (!be_->signal_create_polled(&sig, &val)) break;
        dev_sig_.push_back(sig);
        dev_sig_val_.push_back(val);
      }
      if (dev_sig_.size() != kRecords) {
        for (uint64_t sig : dev_sig_) be_->signal_destroy(sig);
        dev_sig_.clear();
        dev_sig_val_.clear();
      }
    }
    mma_status_t w = warm_up();
    if (w != MMA_OK) return w;
    thread_ = std::thread([this] {
      // Naps of tens of microseconds (see nap): wake within 1 us of the
      // deadline instead of the default 50 us of timer slack.
      prctl(PR_SET_TIMERSLACK, 1000UL, 0UL, 0UL, 0UL);
      loop();
    });
    return MMA_OK;
  }

  // The first command on an engine makes ROCr create that engine's queue
  // (milliseconds); do it here rather than inside the first transfer.
  mma_status_t warm_up() {
    if (paths_.empty()) return MMA_OK;
    void* host = nullptr;
    mma_status_t rc = be_->alloc_host_scratch(4096, &host);
    if (rc != MMA_OK) return rc;
    for (auto& path : paths_) {
      SdmaSlot& s = slots_[path.slots[0]];
      be_->signal_store(s.sig, 1);
      void* stage = reinterpret_cast<void*>(s.staging);
      const bool ok = dir_ == MMA_H2D ? be_->copy(path.engine, stage, true, host, false, 4096, s.sig)
                                      : be_->copy(path.engine, host, false, stage, true, 4096, s.sig);
      if (!ok) {
        rc = fail(MMA_ERR_HSA, "SDMA engine %d rejected a warm-up copy", path.engine);
        break;
      }
      const uint64_t t0 = now_ns();
      int64_t v;
      while ((v = be_->signal_load(s.sig)) > 0 && now_ns() - t0 < 10000000000ull) cpu_relax();
      if (v != 0) {  // still in flight or failed: leave the engine out rather than reuse its signal
        rc = fail(MMA_ERR_HSA, "SDMA engine %d did not complete a warm-up copy", path.engine);
        break;
      }
    }
    be_->free_host_scratch(host);
    return rc;
  }

  // Stops the engine thread and frees what the GPU side shares with it. With
  // release = false (transfers still in flight: a kernel may still read its
  // record, a copy engine still decrement a signal) that memory and those
  // signals are left alone rather than unmapped under them.
  void shutdown(bool release = true) {
    {
      std::lock_guard<std::mutex> g(mu_);
      if (!thread_.joinable()) return;
      stop_ = true;
      stop_flag_ = true;
    }
    cv_.notify_all();
    thread_.join();
    if (!release) {
      slots_.clear();
      dev_sig_.clear();
      dev_sig_val_.clear();
      ds_ = nullptr;
      recs_ = nullptr;
      light_ = nullptr;
      pool_tab_ = nullptr;
      pool_ctr_ = nullptr;
      return;
    }
    for (auto& s : slots_) be_->signal_destroy(s.sig);
    slots_.clear();
    for (uint64_t sig : dev_sig_) be_->signal_destroy(sig);
    dev_sig_.clear();
    dev_sig_val_.clear();
    if (ds_) be_->free_device_state(ds_);
    if (recs_) be_->free_records(recs_);
    if (light_) be_->free_records(light_);
    if (pool_tab_) be_->free_records(pool_tab_);
    if (pool_ctr_) be_->free_device_state(pool_ctr_);
    ds_ = nullptr;
    recs_ = nullptr;
    light_ = nullptr;
    pool_tab_ = nullptr;
    pool_ctr_ = nullptr;
  }

  pthread_t native_handle() { return thread_.native_handle(); }
  uint32_t sdma_mask() const {
    uint32_t m = 0;
    for (auto& p : paths_) m |= 1u << p.engine;
    return m;
  }
  bool moving() const { return moving(now_ns()); }
  bool cu_enabled() const { return (cfg_.mask[dir_] & MMA_PATH_CU) != 0; }
  bool device_control() const { return cfg_.device != 0; }
  // Both directions at once on one link (Section 5.1.2, concurrent flows):
  // the two directions' engines share the copy engines, and each copy engine
  // runs the commands of both directions from one in-order queue. The other
  // direction's commands on a copy engine (peer) are neither foreign work nor
  // congestion: a command of ours only waits behind those that were queued
  // before it. On the mixed workload (a device-to-host KV offload beside a
  // host-to-device weight load, whose merged commands run for milliseconds),
  // counting that wait as congestion backed the offload's engines off about 66
  // times per run (each command 2.3-3.4 ms at the head of this engine's view of
  // the queue, while the other direction's commands ahead of it ran); allowing
  // for the bytes queued ahead at submission, 0-2 times.
  //
  // While the other direction moves, a direction pulls only from its duplex
  // paths (cfg.duplex[dir]): by default the host-facing engines alone for
  // host-to-device, and engines 2-5 alone for device-to-host. No command then
  // waits behind the other direction's merged commands, and neither direction's
  // CU path puts its traffic on the lanes the other one's data uses: CU
  // zero-copy loads send their read requests upstream beside device-to-host
  // data, and CU stores to host memory share those lanes in small writes. On
  // the mixed workload (the 34-group weight load beside the 2048-block offload,
  // streams side by side) that keeps the weight stream within 0.4% of the
  // native schedule (304.3-305.2 ms against 303.4-303.7 ms), with the offload
  // at 102-104 ms; all paths shared: 309-312 and 170-174 ms. The CU path still
  // takes micro-tasks that no other path may carry. Device control has no
  // phases: its copy-engine share stays on the direction's own path mask.
  // Called once both engines are initialised.
  void set_peer(const Engine* peer) { peer_ = peer; }
  // Bytes of the other direction's commands in flight on copy engine e.
  uint64_t peer_bytes_on(int e) const { return peer_ ? peer_->eng_bytes_[e].load(std::memory_order_relaxed) : 0; }
  // The other direction has had a started transfer that is not complete
  // within the last kDuplexHoldNs.
  bool peer_moving(uint64_t now) const { return peer_ && peer_->moving(now); }
  bool moving(uint64_t now) const { return now < moving_until_.load(std::memory_order_relaxed); }

  // Transfers tracked by the submitting threads are in flight (see track).
  bool tracked() const { return n_tracked_.load(std::memory_order_acquire) != 0; }
  bool has_sdma() const { return !paths_.empty(); }
  uint64_t stage_bytes() const { return stage_bytes_; }

  // A transfer that the CU path takes whole (see prepare): it runs as one
  // self-contained launch and needs a light slot, not a record.
  bool whole_eligible(const Transfer* x, uint64_t payload_bytes, bool kv) const {
    if (!cu_enabled() || cfg_.static_split || x->tasks.empty() || payload_bytes > cfg_.whole[dir_]) return false;
    if (kv) return !x->pool_dev && whole_kv_per(x) != 0;
    return x->tasks.size() <= kPrefill;
  }

  // Pieces per CU entry of a whole KV transfer: the engine thread's entry size,
  // grown until all of the transfer's entries fit the launch arguments (one
  // entry never spans two micro-tasks, i.e. two blocks); 0 if they cannot.
  uint64_t whole_kv_per(const Transfer* x) const {
    uint64_t per = std::max<uint64_t>(1, cfg_.sub / x->piece), biggest = 0;
    for (const Task& t : x->tasks) biggest = std::max(biggest, t.bytes);
    for (;;) {
      uint64_t e = 0;
      for (const Task& t : x->tasks) e += (t.bytes + per - 1) / per;
      if (e <= kPrefill) return per;
      if (per >= biggest) return 0;
      per = std::min(biggest, 2 * per);
    }
  }

  // Takes a light slot for a whole transfer, else a record; blocks until one is
  // free (or the timeout passes). Called with the submission mutex held, never
  // by the engine thread. Light slots outnumber records 64 to 1, so a deep
  // queue of small transfers on a stream does not wait for the GPU.
  bool acquire(Transfer* x, uint64_t payload_bytes, bool kv, uint64_t timeout_ms) {
    bool light = whole_eligible(x, payload_bytes, kv);
    reap();
    std::unique_lock<std::mutex> lk(mu_);
    // An HBM pool launch needs room for its table in the arena; without it the
    // transfer takes the ring path like any other.
    if (x->pool_launch) light = x->pool_launch = !g_fault_pool_no_table.load() && take_tab(x);
    std::deque<uint32_t>& pool = light ? free_light_ : free_recs_;
    if (pool.empty() && !wait_for_pool(lk, pool, timeout_ms)) {
      give_tab(x);
      return false;
    }
    const uint32_t i = pool.front();
    pool.pop_front();
    lk.unlock();
    const uint32_t slots = light ? kPrefill : kRingSize;
    x->owner.reset(new int32_t[slots]);
    x->tdone.reset(new uint8_t[slots]);
    if (light) {
      x->light = static_cast<int32_t>(i);
      x->rec = nullptr;
      x->ring = light_ring_.get();
      x->done_host = light_ + static_cast<uint64_t>(i) * kPrefill;
    } else {
      x->rec_idx = i;
      x->rec = &recs_[i];
      x->ring = x->rec->ring;
      x->done_host = x->rec->done;
    }
    return true;
  }
  // Waits (lk held on entry and exit) until `pool` has a free entry. Slots of
  // transfers that the submitting threads track themselves (track) come back
  // only when one of them reaps, so this thread reaps while it waits.
  bool wait_for_pool(std::unique_lock<std::mutex>& lk, const std::deque<uint32_t>& pool, uint64_t timeout_ms) {
    const auto deadline = std::chrono::steady_clock::now() + std::chrono::milliseconds(timeout_ms);
    while (pool.empty()) {
      if (std::chrono::steady_clock::now() >= deadline) return false;
      lk.unlock();
      reap();
      lk.lock();
      if (!pool.empty()) break;
      cv_done_.wait_for(lk, std::chrono::microseconds(20));
    }
    return true;
  }

  void release_unused(Transfer* x) {
    std::lock_guard<std::mutex> g(mu_);
    give_tab(x);
    if (x->light >= 0)
      free_light_.push_back(static_cast<uint32_t>(x->light));
    else
      free_recs_.push_back(x->rec_idx);
    cv_done_.notify_all();
  }
  // Table arena segments for an HBM pool launch (mu_ held): the first run of
  // free segments that holds the table, or false if there is none.
  bool take_tab(Transfer* x) {
    if (!pool_tab_) return false;
    const uint64_t need = (x->pool_pairs.size() + kPoolTabSeg - 1) / kPoolTabSeg;
    if (need == 0 || need > seg_used_.size()) return false;
    for (size_t i = 0, run = 0; i < seg_used_.size(); ++i) {
      run = seg_used_[i] ? 0 : run + 1;
      if (run == need) {
        const size_t first = i + 1 - need;
        std::fill(seg_used_.begin() + static_cast<long>(first), seg_used_.begin() + static_cast<long>(i) + 1, 1);
        x->tab_seg = static_cast<int32_t>(first);
        x->tab_nseg = static_cast<uint32_t>(need);
        return true;
      }
    }
    return false;
  }
  void give_tab(Transfer* x) {  // mu_ held
    if (x->tab_seg < 0) return;
    std::fill(seg_used_.begin() + x->tab_seg, seg_used_.begin() + x->tab_seg + x->tab_nseg, 0);
    x->tab_seg = -1;
    x->tab_nseg = 0;
  }
  Record* rec_dev(uint32_t i) const { return recs_dev_ + i; }
  DevState* ds(uint32_t i) const { return ds_ + i; }

  // CU path's first pulls, made before the transfer is handed to the engine
  // thread (no concurrent access to x yet): the dummy task's workers can start
  // copying as soon as the stream reaches them, without a host round trip.
  // While the other direction moves, only micro-tasks that the CU path alone
  // may carry (see set_peer).
  void prefill(Transfer* x) { pull_cu(x, cu_paused_at(now_ns())); }

  // Workgroups of the dummy-task kernel: one wave per ring entry that can be
  // outstanding at once (waves beyond that would only poll host memory, and
  // every poll is a PCIe read that competes with the payload).
  // x-packed KV pieces: a wave alternates between reading a head group into its
  // LDS tile and writing it out, with no reads in flight during the second
  // phase, so more waves are needed for the same bytes in flight.
  uint32_t grid_for(uint64_t bytes, uint64_t sub, bool needs_cu, bool staged, bool pool_dev, bool wide) const {
    if (!needs_cu) return 1;
    if (pool_dev) {  // HBM gather/scatter: as many waves as there are micro-tasks, up to the limit
      const uint64_t tasks = (bytes + cfg_.chunk - 1) / cfg_.chunk;
      return static_cast<uint32_t>(std::max<uint64_t>(1, std::min<uint64_t>((tasks + 3) / 4, kMaxWorkgroups)));
    }
    const uint64_t total = (bytes + sub - 1) / sub;
    const uint64_t per_task = (cfg_.chunk + sub - 1) / sub;
    // Entries in flight with a phase's paths (the direction's own, or its
    // duplex paths while the other direction moves; see set_peer): the CU
    // path's depth, and for staged transfers each engine's staging.
    const auto inflight_with = [&](uint32_t paths) {
      uint64_t f = (paths & MMA_PATH_CU) && cu_enabled() ? cfg_.cu_depth * per_task : 0;
      if (staged) f += static_cast<uint64_t>(__builtin_popcount(paths & sdma_mask())) * cfg_.depth * per_task;
      return f;
    };
    const uint64_t inflight = std::max(inflight_with(cfg_.mask[dir_]), inflight_with(cfg_.duplex[dir_]));
    uint64_t g = (std::max<uint64_t>(1, std::min(total, inflight)) + kWavesPerWG - 1) / kWavesPerWG;
    g = std::max<uint64_t>(1, std::min<uint64_t>(g, wg_cap(wide)));
    return static_cast<uint32_t>(g);
  }

  // Workgroup limit of one launch. x-packed and head-major launches (their
  // waves move 8 KiB per batch through 16-byte units, against the plain copy's
  // two 16 KiB batches) get 1.5x cu_workgroups. For x-packed,
  // on the 64k-token workload (fetch / offload GB/s at the default 16) 16
  // workgroups gave 54.6 / 49.1, 20 gave 57.27 / 56.93, 24 gave 57.33 / 56.85,
  // 28 gave 57.14 / 56.82, 32 gave 56.97 / 56.42, 40 and 48 gave 56.4 and 55.8
  // on the fetch: past about 24, the waves' polls and LDS phases cost more
  // than their extra reads in flight gain.
  uint64_t wg_cap(bool wide) const {
    const uint64_t w = wide ? (3ull * cfg_.cu_wgs + 1) / 2 : cfg_.cu_wgs;
    return std::min<uint64_t>(w, kMaxWorkgroups);
  }

  // Everything between the plan and the kernel launch, for a transfer that
  // holds a record: epoch, static-split flags, CU entry size, grid, the CU
  // path's first pulls, the self-contained decision and the kernel
  // arguments. Returns the grid in workgroups.
  uint32_t prepare(Transfer* x, uint64_t seq, uint64_t payload_bytes, const KvGeom* kv, uint64_t watchdog_ticks,
                   KernelArgs& a) {
    x->claimed.assign(x->tasks.size(), 0);
    x->left.assign(x->tasks.size(), 0);
    x->seq = seq;
    x->t_submit = now_ns();
    x->bytes = payload_bytes;
    if (Record* r = x->rec) {
      r->h.seq = x->seq;
      r->h.status = 0;
      __atomic_thread_fence(__ATOMIC_RELEASE);
    }
    if (x->pool_launch) return prepare_pool(x, kv, a);
    if (cfg_.static_split && has_sdma() && x->sdma_ok) {
      for (size_t i = 0; i < x->tasks.size(); ++i) {
        uint32_t& f = x->tasks[i].flags;
        if (f & kPlanCuOnly) continue;
        f |= static_cu_task(i, cfg_.static_cu_percent) ? kPlanCuOnly : kPlanSdmaOnly;
      }
    }
    x->cu_only_left = static_cast<size_t>(std::count_if(
        x->tasks.begin(), x->tasks.end(), [](const Task& t) { return (t.flags & kPlanCuOnly) != 0; }));
    const bool staged = x->kind != Kind::kLinear && has_sdma() && x->sdma_ok;
    const bool needs_cu = cu_enabled() || staged ||
                          std::any_of(x->tasks.begin(), x->tasks.end(),
                                      [](const Task& t) { return (t.flags & kPlanCuOnly) != 0; });
    // CU ring entries of a linear transfer are cu_sub_bytes. A transfer of at
    // most cfg.whole[dir] bytes whose micro-tasks can all travel in the launch's
    // arguments (at most kPrefill entries) is taken whole by the CU path, each
    // micro-task cut into at most kPrefill / tasks entries of whole 16 KiB steps
    // (one wave register batch): the kernel is then the transfer's only copy
    // engine and needs no host round trip at all -- no start signal, no ring, no
    // wait for `complete` -- which at these sizes is worth more than the copy
    // engines' slightly better link efficiency. Otherwise a transfer that fits
    // the prefilled entries is still cut into 16 KiB steps, so that more waves
    // share it.
    x->sub = cfg_.sub;
    if (kv && x->light >= 0) {  // a whole KV transfer (acquire gave it a light slot)
      x->kv_per = whole_kv_per(x);
      x->whole = true;
    } else if (!kv && whole_eligible(x, payload_bytes, false)) {
      const uint64_t per_task = kPrefill / x->tasks.size();
      uint64_t biggest = 0;
      for (const Task& t : x->tasks) biggest = std::max(biggest, t.bytes);
      const uint64_t sub = (biggest + per_task - 1) / per_task;
      x->sub = std::max<uint64_t>(kSmallSub, (sub + kSmallSub - 1) / kSmallSub * kSmallSub);
      x->whole = true;
    } else if (!kv && payload_bytes <= kPrefill * cfg_.sub) {
      const uint64_t per = (payload_bytes + kPrefill - 1) / kPrefill;
      x->sub = std::min<uint64_t>(cfg_.sub,
                                  std::max<uint64_t>(kSmallSub, (per + kSmallSub - 1) / kSmallSub * kSmallSub));
    }
    uint32_t grid = grid_for(payload_bytes, x->sub, needs_cu || x->pool_dev, staged, x->pool_dev,
                             kv && kv->layout != kKvLayoutPiece);
    x->waves = grid * kWavesPerWG;
    prefill(x);
    const uint32_t n_pre =
        kv && !x->whole ? 0u : static_cast<uint32_t>(std::min<uint64_t>(x->pushed, kPrefill));
    // Everything fits the launch: all tasks were claimed by the CU prefill (so no
    // copy engine can take part) and all their entries are in the kernel args.
    // One wave per entry; the engine treats the transfer as started.
    x->self_contained = (!kv || x->whole) && x->n_claimed == x->tasks.size() && x->pushed == n_pre;
    if (x->self_contained) {
      grid = (n_pre + kWavesPerWG - 1) / kWavesPerWG;
      x->waves = grid * kWavesPerWG;
      x->started = true;
      x->t_started = x->t_submit;
    }
    if (x->light >= 0) {  // whole, hence self-contained: nothing to close or publish in a record
      x->closed = x->completed = true;
      x->t_complete = x->t_submit;
    }
    fill_args(x, kv, n_pre, grid, watchdog_ticks, a);
    return grid;
  }

  // An HBM pool launch: the table goes to the arena, the grid is sized to
  // the spans (whole pieces for head-major blocks; at least one per wave, at
  // most kPoolMaxWorkgroups workgroups),
  // and the kernel is the transfer's only copy engine. Returns the grid.
  uint32_t prepare_pool(Transfer* x, const KvGeom* kv, KernelArgs& a) {
    const uint64_t nblk = x->pool_pairs.size();
    memcpy(pool_tab_ + static_cast<uint64_t>(x->tab_seg) * kPoolTabSeg, x->pool_pairs.data(),
           nblk * sizeof(uint64_t));
    __atomic_thread_fence(__ATOMIC_RELEASE);
    std::fill(x->claimed.begin(), x->claimed.end(), 1);
    x->n_claimed = x->tasks.size();
    x->pushed = 1;
    x->whole = x->self_contained = true;
    x->started = x->closed = x->completed = true;
    x->t_started = x->t_complete = x->t_submit;
    const uint64_t spans = kv->layout == kKvLayoutHnd ? 1 : (kv->piece + kPoolSpan - 1) / kPoolSpan;
    const uint64_t units = nblk * 2 * kv->layers * spans;
    uint64_t grid = std::min<uint64_t>(kPoolMaxWorkgroups, (units + kWavesPerWG - 1) / kWavesPerWG);
    const uint64_t per_wg = (units + grid - 1) / grid;
    grid = (units + per_wg - 1) / per_wg;
    x->waves = static_cast<uint32_t>(grid) * kWavesPerWG;
    fill_args(x, kv, 0, static_cast<uint32_t>(grid), 0, a);
    a.self_contained = 1;
    a.pool_tab = pool_tab_dev_ + static_cast<uint64_t>(x->tab_seg) * kPoolTabSeg;
    a.pool_ctr = pool_ctr_ + x->light;
    a.pool_base = x->pool_base;
    a.pool_units = units;
    a.pool_per_wg = per_wg;
    a.pool_spans = static_cast<uint32_t>(spans);
    a.pool_to_paged = x->kind == Kind::kKvFetch ? 1u : 0u;
    return static_cast<uint32_t>(grid);
  }

  // Kernel arguments common to both control modes.
  void fill_args(const Transfer* x, const KvGeom* kv, uint32_t n_pre, uint32_t grid, uint64_t watchdog_ticks,
                 KernelArgs& a) const {
    memset(&a, 0, offsetof(KernelArgs, layer_ptr));
    a.n_pre = n_pre;
    a.self_contained = x->self_contained ? 1u : 0u;
    for (uint32_t t = 0; t < n_pre; ++t) {
      const CuEntry& en = x->ring[t];
      a.pre[t][0] = en.a;
      a.pre[t][1] = en.b;
      a.pre[t][2] = static_cast<uint64_t>(en.count) | (static_cast<uint64_t>(en.kind_p0) << 32);
    }
    if (kv) {
      a.kv_piece_bytes = kv->piece;
      a.kv_kstride = kv->kstride;
      a.kv_layers = kv->layers;
      a.kv_layout = kv->layout;
      a.kv_tokens = kv->tokens;
      a.kv_heads = kv->heads;
      a.kv_row_bytes = kv->row_bytes;
      a.kv_elem = kv->elem;
      a.kv_lds_wave = kv->lds_wave;
      memcpy(a.layer_ptr, kv->layer_ptr, sizeof(uint64_t) * kv->layers);
    }
    if (x->light >= 0) {
      a.rec = nullptr;
      a.ds = nullptr;
      a.done = light_dev_ + static_cast<uint64_t>(x->light) * kPrefill;
    } else {
      a.rec = rec_dev(x->rec_idx);
      a.ds = ds(x->rec_idx);
      a.done = a.rec->done;
    }
    a.seq = x->seq;
    a.watchdog_ticks = watchdog_ticks;
    a.total_waves = grid * kWavesPerWG;
    a.release_each = x->dir == MMA_D2H ? 1u : 0u;
  }

  // ---------------------------------------------------------------- device control
  // A control plane with no host thread in the loop -- the direction Section 6
  // (Current limitations) gives for the cost of a CPU-driven control plane on
  // fine-grained transfers. The submitting thread plans the whole transfer
  // before the launch:
  //   - the CU path's share goes into the record's ring in full, so the
  //     kernel's waves claim every entry with their device atomic and nothing
  //     is ever appended later;
  //   - on a stream with nothing pending, a fixed share of a linear transfer
  //     (the last 100 - device_cu_percent % of its bytes) goes to the copy
  //     engines at once, split between them, all commands counting down one
  //     polled completion signal.
  // The kernel's last wave waits for that signal instead of the engine
  // thread's `complete` word, and the submitting thread recycles the record
  // once the kernel has released it (reap). Against the engine thread
  // this gives up pulling and back-off on the copy engines, whose share is
  // fixed at submission, and copy engines on a stream with work pending: a
  // command that waited for the stream would hold the head of the engine's
  // in-order queue, which every other copy of the process shares. KV
  // transfers run on the CU path alone (their copy-engine share would need
  // staging slots recycled between commands). Returns the grid, or 0 if the
  // transfer has more micro-tasks than the ring has entries; the caller then
  // hands it to the engine thread.
  uint32_t prepare_device(Transfer* x, uint64_t seq, uint64_t payload_bytes, const KvGeom* kv,
                          uint64_t watchdog_ticks, bool stream_idle, KernelArgs& a) {
    const size_t n = x->tasks.size();
    if (n == 0 || n > kRingSize || !x->rec) return 0;
    const bool linear = x->kind == Kind::kLinear;
    // CU entry size: the engine thread's, grown until every micro-task would
    // fit the ring, so that the tasks of a command the runtime refuses can
    // still go to the CU path.
    uint64_t per, biggest = 0;
    for (const Task& t : x->tasks) biggest = std::max(biggest, t.bytes);
    if (linear) {
      per = cfg_.sub;
      if (payload_bytes <= kPrefill * cfg_.sub) {
        const uint64_t p = (payload_bytes + kPrefill - 1) / kPrefill;
        per = std::min<uint64_t>(cfg_.sub, std::max<uint64_t>(kSmallSub, (p + kSmallSub - 1) / kSmallSub * kSmallSub));
      }
    } else {
      per = x->pool_dev ? biggest : std::max<uint64_t>(1, cfg_.sub / x->piece);
    }
    auto entries = [&](uint64_t p) {
      uint64_t e = 0;
      for (const Task& t : x->tasks) e += (t.bytes + p - 1) / p;
      return e;
    };
    while (per < biggest && entries(per) > kRingSize) per = std::min(biggest, 2 * per);
    if (entries(per) > kRingSize) return 0;
    if (linear)
      x->sub = per;
    else
      x->kv_per = per;

    x->claimed.assign(n, 0);
    x->left.assign(n, 0);
    x->dev_path.assign(n, static_cast<uint8_t>(MMA_NUM_PATHS - 1));
    x->seq = seq;
    x->t_submit = x->t_started = now_ns();
    x->bytes = payload_bytes;
    x->started = x->closed = true;
    Record* r = x->rec;
    r->h.seq = seq;
    r->h.status = 0;
    __atomic_thread_fence(__ATOMIC_RELEASE);

    // The copy engines' share: the last micro-tasks, by bytes, on the
    // engines of the direction's own path mask (its duplex-only engines are
    // for the engine thread's phases; see set_peer).
    std::vector<int> dev_paths;
    for (size_t k = 0; k < paths_.size(); ++k)
      if ((cfg_.mask[dir_] >> paths_[k].engine) & 1u) dev_paths.push_back(static_cast<int>(k));
    std::vector<size_t> eng_tasks;
    if (stream_idle && linear && x->sdma_ok && !dev_sig_.empty() && !dev_paths.empty()) {
      const uint64_t cu_pct = cu_enabled() ? cfg_.device_cu_percent : 0;
      const uint64_t want = payload_bytes / 100 * (100 - cu_pct) + payload_bytes % 100 * (100 - cu_pct) / 100;
      uint64_t got = 0;
      for (size_t i = n; i-- > 0 && got < want;) {
        if (x->tasks[i].flags & kPlanCuOnly) continue;
        eng_tasks.push_back(i);
        got += x->tasks[i].bytes;
      }
      std::reverse(eng_tasks.begin(), eng_tasks.end());
      for (size_t i : eng_tasks) x->claimed[i] = 1;
    }
    // The CU path's share, in task order.
    x->pushed = 0;
    for (size_t i = 0; i < n; ++i)
      if (!x->claimed[i]) push_device(x, i);
    // Engine k of dev_paths takes the engine tasks whose first byte falls in
    // the k-th equal part of their bytes; runs that follow each other in both
    // address spaces go as one command.
    struct Cmd {
      int path;
      size_t first, end;
      uint64_t bytes;
    };
    std::vector<Cmd> cmds;
    uint64_t total = 0, at = 0;
    for (size_t i : eng_tasks) total += x->tasks[i].bytes;
    for (size_t k = 0; k < eng_tasks.size(); ++k) {
      const size_t i = eng_tasks[k];
      const Task& t = x->tasks[i];
      const int path = dev_paths[at * dev_paths.size() / std::max<uint64_t>(total, 1)];
      at += t.bytes;
      if (!cmds.empty()) {
        Cmd& c = cmds.back();
        const Task& prev = x->tasks[c.end - 1];
        if (c.path == path && c.end == i && t.src_dma == prev.src_dma + prev.bytes &&
            t.dst_dma == prev.dst_dma + prev.bytes) {
          c.end = i + 1;
          c.bytes += t.bytes;
          continue;
        }
      }
      cmds.push_back(Cmd{path, i, i + 1, t.bytes});
    }
    const uint64_t sig = cmds.empty() ? 0 : dev_sig_[x->rec_idx];
    if (!cmds.empty()) {
      uint64_t f = g_fault_signal_hold.load();
      while (f > 0 && !x->dev_hold)
        if (g_fault_signal_hold.compare_exchange_weak(f, f - 1)) x->dev_hold = true;
      be_->signal_store(sig, static_cast<int64_t>(cmds.size()) + (x->dev_hold ? 1 : 0));
    }
    const bool h2d = dir_ == MMA_H2D;
    for (const Cmd& c : cmds) {
      const Task& t = x->tasks[c.first];
      bool ok = true;
      uint64_t f = g_fault_submit_fail.load();
      while (ok && f > 0)
        if (g_fault_submit_fail.compare_exchange_weak(f, f - 1)) ok = false;
      ok = ok && be_->copy(paths_[c.path].engine, reinterpret_cast<void*>(t.dst_dma), h2d,
                           reinterpret_cast<void*>(t.src_dma), !h2d, c.bytes, sig);
      if (ok) {
        st_->sdma_commands += 1;
        if (!x->t_first_sdma) x->t_first_sdma = now_ns();
        for (size_t i = c.first; i < c.end; ++i) x->dev_path[i] = static_cast<uint8_t>(paths_[c.path].engine);
      } else {
        // Refused: its tasks go to the CU path (the ring has room for them).
        st_->submit_failures += 1;
        be_->signal_sub(sig, 1);
        for (size_t i = c.first; i < c.end; ++i) push_device(x, i);
      }
    }
    x->dev_cmds = static_cast<uint32_t>(cmds.size());

    uint32_t grid;
    if (x->pool_dev) {
      grid = grid_for(payload_bytes, x->sub, true, false, true, false);
    } else {
      const uint64_t cap = wg_cap(kv && kv->layout != kKvLayoutPiece);
      grid = static_cast<uint32_t>(
          std::max<uint64_t>(1, std::min<uint64_t>((x->pushed + kWavesPerWG - 1) / kWavesPerWG, cap)));
    }
    x->waves = grid * kWavesPerWG;
    const uint32_t n_pre = kv ? 0u : static_cast<uint32_t>(std::min<uint64_t>(x->pushed, kPrefill));
    fill_args(x, kv, n_pre, grid, watchdog_ticks, a);
    a.device_ctl = 1;
    a.n_total = static_cast<uint32_t>(x->pushed);
    a.sdma_left = x->dev_cmds ? dev_sig_val_[x->rec_idx] : nullptr;
    return grid;
  }

  // A launched transfer that needs no engine-thread work -- every transfer
  // under device control, and a whole transfer in a light slot in either mode
  // (the kernel is its only copy engine) -- is tracked by the submitting
  // threads until reap retires it; the engine thread is not woken for it.
  void track(std::unique_ptr<Transfer> x) {
    {
      std::lock_guard<std::mutex> g(mu_);
      ++inflight_;
    }
    std::lock_guard<std::mutex> g(dev_mu_);
    tracked_.push_back(std::move(x));
    n_tracked_.fetch_add(1, std::memory_order_release);
  }

  // Device control: the dummy-task launch failed after the copy engines were
  // given their share. Waits for them (they write the caller's buffers), then
  // frees the record; one that does not drain is never reused.
  void abandon_device(Transfer* x, uint64_t timeout_ms) {
    if (x->dev_cmds) {
      const uint64_t sig = dev_sig_[x->rec_idx];
      if (x->dev_hold) {
        be_->signal_sub(sig, 1);
        x->dev_hold = false;
      }
      const uint64_t t0 = now_ns();
      while (be_->signal_load(sig) > 0) {
        if (now_ns() - t0 > timeout_ms * 1000000ull) return;
        std::this_thread::sleep_for(std::chrono::microseconds(20));
      }
    }
    release_unused(x);
  }

  // Retires tracked transfers whose kernel has finished with their record or
  // light slot (and whose copy-engine commands have all landed, even after a
  // watchdog). Any thread may call it. Only the oldest kReapWindow transfers
  // are looked at, so a deep queue costs each submission a bounded scan;
  // transfers on one stream finish in order, so the oldest go first.
  void reap() {
    if (!tracked()) return;
    std::lock_guard<std::mutex> g(dev_mu_);
    for (size_t k = 0; k < tracked_.size() && k < kReapWindow;) {
      Transfer* x = tracked_[k].get();
      if (!tracked_done(x)) {
        ++k;
        continue;
      }
      bool bad = false;
      if (x->rec) bad = ld_acq(&x->rec->h.status) != 0;
      if (x->dev_cmds && be_->signal_load(dev_sig_[x->rec_idx]) < 0) bad = true;
      x->t_last_task = x->t_complete = now_ns();
      for (size_t i = 0; i < x->tasks.size(); ++i) {
        const int path = x->dev_path.empty() ? MMA_NUM_PATHS - 1 : x->dev_path[i];
        const Task& t = x->tasks[i];
        st_->path_bytes[path] += x->kind == Kind::kLinear ? t.bytes : t.bytes * x->piece;
        st_->path_tasks[path] += 1;
        ++x->path_tasks[path];
      }
      x->n_done = x->tasks.size();
      finish(x, bad, true);
      tracked_.erase(tracked_.begin() + static_cast<long>(k));
      n_tracked_.fetch_sub(1, std::memory_order_release);
    }
  }

  void submit(std::unique_ptr<Transfer> x) {
    bool wake;
    {
      std::lock_guard<std::mutex> g(mu_);
      incoming_.push_back(std::move(x));
      ++inflight_;
      wake = engine_waiting_;
    }
    n_incoming_.fetch_add(1, std::memory_order_release);
    if (wake) cv_.notify_all();  // the engine thread sleeps after 2 ms without work, or naps
  }

  bool wait_idle(uint64_t timeout_ms) {
    const auto deadline = std::chrono::steady_clock::now() + std::chrono::milliseconds(timeout_ms);
    for (;;) {
      reap();
      std::unique_lock<std::mutex> lk(mu_);
      if (inflight_ == 0) return true;
      if (std::chrono::steady_clock::now() >= deadline) return false;
      if (tracked())
        cv_done_.wait_for(lk, std::chrono::microseconds(50));
      else
        cv_done_.wait_until(lk, deadline);
    }
  }

 private:
  // ---------------------------------------------------------------- ring
  // Append the ring entries of one unit of work. `a` is the contiguous side
  // (linear: source; KV: host or staging range), `b` the other side (linear:
  // destination; KV: GPU block). Returns the number appended, 0 if no room.
  uint32_t push_unit(Transfer* x, int32_t owner, uint32_t kind, uint64_t a, uint64_t b, uint64_t count,
                     uint32_t p0) {
    uint64_t per;
    if ((kind & kEntryKindMask) == kEntryCopy) {
      per = x->sub;
    } else {
      // A wave's ring entry carries cu_sub_bytes of pieces across PCIe (more for
      // a whole transfer, whose entries must fit the launch); for an
      // HBM-resident pool (latency ~1 us instead of several) a whole micro-task.
      per = x->kv_per ? x->kv_per : x->pool_dev ? count : std::max<uint64_t>(1, cfg_.sub / x->piece);
    }
    const uint64_t ne = (count + per - 1) / per;
    // Keep one slot per wave free for the end markers written at close.
    if (x->pushed + ne - x->done_upto > kRingSize - x->waves) return 0;
    return append(x, owner, kind, a, b, count, p0, per);
  }

  // Appends the entries of one unit of work, `per` bytes (linear) or pieces
  // (KV) each; the caller has checked that they fit the ring.
  uint32_t append(Transfer* x, int32_t owner, uint32_t kind, uint64_t a, uint64_t b, uint64_t count, uint32_t p0,
                  uint64_t per) {
    const uint64_t ne = (count + per - 1) / per;
    for (uint64_t k = 0; k < ne; ++k) {
      const uint64_t t = x->pushed++;
      const uint32_t slot = static_cast<uint32_t>(t % kRingSize);
      const uint64_t c = std::min(per, count - k * per);
      CuEntry* e = &x->ring[slot];
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
    x->done_bytes += bytes;
    st_->path_bytes[path_stat] += bytes;
    st_->path_tasks[path_stat] += 1;
    x->progress = true;
  }

  bool scan_cu(Transfer* x) {
    bool p = false;
    for (uint64_t t = x->done_upto; t < x->pushed; ++t) {
      const uint32_t slot = static_cast<uint32_t>(t % kRingSize);
      if (x->tdone[slot]) continue;
      if (ld_acq(&x->done_host[slot]) != make_tag(x->seq, t)) continue;
      x->tdone[slot] = 1;
      p = true;
      const int32_t own = x->owner[slot];
      if (own >= 0) {
        --x->cu_entries;
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

  // Device control: all CU ring entries of micro-task i (prepare_device has
  // sized them so that every task fits the ring).
  void push_device(Transfer* x, size_t i) {
    const Task& t = x->tasks[i];
    if (x->kind == Kind::kLinear)
      append(x, static_cast<int32_t>(i), kEntryCopy, t.src_cu, t.dst_cu, t.bytes, 0, x->sub);
    else
      append(x, static_cast<int32_t>(i), x->kind == Kind::kKvFetch ? kEntryToPaged : kEntryFromPaged, t.host_cu,
             t.blk, t.bytes, t.p0, x->kv_per);
    x->claimed[i] = 1;
    x->dev_path[i] = static_cast<uint8_t>(MMA_NUM_PATHS - 1);
  }

  // A tracked transfer's kernel is done with its record or light slot.
  bool tracked_done(Transfer* x) {
    if (x->light >= 0) {  // a whole transfer: every entry's done tag is in
      for (uint64_t t = 0; t < x->pushed; ++t)
        if (ld_acq(&x->done_host[t]) != make_tag(x->seq, t)) return false;
      return true;
    }
    if (ld_acq(&x->rec->h.released) != x->seq) return false;
    if (x->dev_hold) {  // the kernel has left: take back the count the fault added
      be_->signal_sub(dev_sig_[x->rec_idx], 1);
      x->dev_hold = false;
    }
    return !x->dev_cmds || be_->signal_load(dev_sig_[x->rec_idx]) <= 0;
  }

  // Outcome, trace and waiter of a retired transfer; frees its record or light slot.
  void finish(Transfer* x, bool bad, bool counted) {
    if (bad) {
      g_sticky.store(1);
      st_->failed += 1;
    }
    if (counted) st_->transfers += 1;
    if (x->pool_launch) st_->pool_launches += 1;
    if (g_trace.load(std::memory_order_relaxed)) record_trace(x, bad);
    if (x->waiter) {
      std::lock_guard<std::mutex> g(x->waiter->mu);
      x->waiter->done = true;
      x->waiter->failed = bad;
      x->waiter->cv.notify_all();
    }
    {
      std::lock_guard<std::mutex> g(mu_);
      give_tab(x);
      if (x->light >= 0)
        free_light_.push_back(static_cast<uint32_t>(x->light));
      else
        free_recs_.push_back(x->rec_idx);
      --inflight_;
    }
    cv_done_.notify_all();
  }

  // ---------------------------------------------------------------- CU path
  bool pull_cu(Transfer* x, bool cu_paused) {
    if (x->failed || x->ignored || x->aborting) return false;
    const bool any = cu_enabled() || x->pool_dev;
    // While the CU path pauses for the other direction (see set_peer), it
    // takes only the micro-tasks no other path may carry.
    const bool paused = cu_paused && !x->pool_dev && !x->whole;
    if (paused && x->cu_only_left == 0) return false;
    // An HBM-resident pool keeps every wave busy: two micro-tasks per wave outstanding.
    const uint32_t depth = x->whole ? ~0u : (x->pool_dev ? 2 * x->waves : cfg_.cu_depth);
    bool p = false;
    while (true) {
      if (x->cu_busy >= depth) x->cu_full = true;
      if (x->cu_full && x->cu_busy < std::min(cfg_.cu_backoff ? cfg_.cu_backoff : depth, depth)) x->cu_full = false;
      if (x->cu_full) break;
      size_t i = x->cur_cu;
      while (i < x->tasks.size() && (x->claimed[i] || (x->tasks[i].flags & kPlanSdmaOnly) ||
                                      (!any && !(x->tasks[i].flags & kPlanCuOnly))))
        ++i;
      x->cur_cu = i;
      if (paused) {  // the cursor above stays where the CU path resumes
        i = std::max(x->cur_cu_only, i);
        while (i < x->tasks.size() && (x->claimed[i] || !(x->tasks[i].flags & kPlanCuOnly))) ++i;
        x->cur_cu_only = i;
      }
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
      if (t.flags & kPlanCuOnly) --x->cu_only_left;
      x->left[i] = ne;
      x->cu_entries += ne;
      ++x->cu_busy;
      p = true;
    }
    return p;
  }

  // ---------------------------------------------------------------- SDMA path
  static bool engine_op(const SdmaSlot& s) { return s.state == kCopy || s.state == kH2DStage || s.state == kD2HStage; }
  int engine_ops(const SdmaPath& path) const {
    int n = 0;
    for (int id : path.slots) n += engine_op(slots_[id]) ? 1 : 0;
    return n;
  }

  bool sdma_copy(SdmaSlot& s, void* dst, bool dst_on_device, const void* src, bool src_on_device, uint64_t bytes) {
    uint64_t f = g_fault_submit_fail.load();
    while (f > 0) {
      if (g_fault_submit_fail.compare_exchange_weak(f, f - 1)) return false;
    }
    if (!s.x->t_first_sdma) s.x->t_first_sdma = now_ns();
    s.t_submit = now_ns();
    s.op_bytes = bytes;
    s.ahead = peer_bytes_on(paths_[s.path].engine);
    SdmaPath& path = paths_[s.path];
    if (engine_ops(path) == 0) path.t_head = s.t_submit;  // (s is not in an engine state yet)
    be_->signal_store(s.sig, 1);
    // counted before the command is queued, so that the other direction never
    // sees the engine in use with none of these bytes on it
    eng_bytes_[path.engine].fetch_add(bytes, std::memory_order_relaxed);
    const bool ok = be_->copy(path.engine, dst, dst_on_device, src, src_on_device, bytes, s.sig);
    if (ok)
      st_->sdma_commands += 1;
    else
      eng_bytes_[path.engine].fetch_sub(bytes, std::memory_order_relaxed);
    return ok;
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
      if (sdma_copy(s, reinterpret_cast<void*>(t.host_dma), false, reinterpret_cast<void*>(s.staging), true,
                    s.count * x->piece)) {
        s.state = kD2HStage;
      } else {
        // The copy engine refused the command. The source blocks are untouched, so the
        // micro-tasks go back to the queue for the CU path, which moves them straight to
        // host memory; the ring is still open for them (this slot kept it open).
        st_->submit_failures += 1;
        requeue_cu(x, s.task, s.task_end);
        free_slot(s);
      }
      --x->sdma_cu_pending;
    }
  }

  // Micro-tasks [i, end) of x go back to the queue, CU path only.
  void requeue_cu(Transfer* x, size_t i, size_t end) {
    for (size_t j = i; j < end; ++j) {
      x->claimed[j] = 0;
      x->tasks[j].flags = (x->tasks[j].flags & ~kPlanSdmaOnly) | kPlanCuOnly;
    }
    x->n_claimed -= end - i;
    x->cu_only_left += end - i;
    x->cur_cu_only = std::min(x->cur_cu_only, i);
    x->cur_cu = std::min(x->cur_cu, i);
    x->progress = true;
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
    if (s.state == kH2DScatterPush) {
      s.state = kH2DScatter;
      --x->sdma_cu_pending;
    } else {
      s.state = kD2HGather;  // still pending until its copy-engine command is accepted
    }
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
          if (s.state == kD2HGather) --s.x->sdma_cu_pending;
          free_slot(s);
          p = true;
        }
        continue;
      }
      if (!engine_op(s)) continue;
      const int64_t v = be_->signal_load(s.sig);
      if (v > 0) continue;
      p = true;
      Transfer* x = s.x;
      x->progress = true;
      // The engine runs our commands in order: the next one is at the head now.
      SdmaPath& path = paths_[s.path];
      const uint64_t now = now_ns(), start = std::max(path.t_head, s.t_submit);
      if (v == 0 && now > start && s.op_bytes >= kRateMinBytes) {
        const double obs = static_cast<double>(now - start) / static_cast<double>(s.op_bytes);
        path.ns_per_byte = path.ns_per_byte > 0 ? 0.75 * path.ns_per_byte + 0.25 * obs : obs;
      }
      path.t_head = now;
      eng_bytes_[paths_[s.path].engine].fetch_sub(s.op_bytes, std::memory_order_relaxed);
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
  // KV block's consecutive pieces that fit the staging slot), `cap` micro-tasks
  // at most. Each ROCr copy command costs about 8 us of engine time (measured),
  // so at small chunk sizes one command per micro-task would cap an engine well
  // below the link.
  size_t merge_run(const Transfer* x, size_t i, size_t cap) const {
    const bool sdma_only = (x->tasks[i].flags & kPlanSdmaOnly) != 0;
    uint64_t total = x->tasks[i].bytes;
    size_t j = i + 1;
    for (; j < x->tasks.size() && j - i < cap; ++j) {
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

  // Micro-tasks of x that copy-engine `path` may still take: each engine holds
  // at most an equal share, among the engines, of the work of x not yet landed
  // (claimed-but-outstanding plus unclaimed). Early in a transfer the share is
  // large, so an engine gets few long commands and ROCr's per-command cost is
  // paid rarely; it shrinks as the transfer drains, so the engines finish
  // together (guided self-scheduling, Polychronopoulos and Kuck, 1987,
  // extended to paths with several commands in flight). The CU path is not
  // counted: it pulls 64 KiB ring entries at its own depth, fills whatever the
  // engines leave, and strands no work at the end. An idle engine always gets
  // at least one micro-task.
  size_t fair_share(const Transfer* x, const SdmaPath& path) const {
    const size_t unclaimed = x->tasks.size() - x->n_claimed;
    const size_t outstanding = x->n_claimed - x->n_done;
    size_t mine = 0;
    for (int id : path.slots) {
      const SdmaSlot& s = slots_[id];
      if (s.x == x && s.state != kFree) mine += s.task_end - s.task;
    }
    const size_t n = std::max<size_t>(1, n_pull_paths_);
    const size_t fair = (unclaimed + outstanding + n - 1) / n;
    return fair > mine ? fair - mine : 0;
  }

  // A path is overdue when its oldest command has been at the head of the
  // engine's queue for four times what its size needs at an equal share of a
  // 50 GB/s link (overdue_gbs) among all paths, plus 0.5 ms of slack. (Timing
  // from submission would count the wait behind the path's own earlier commands.)
  bool overdue(const SdmaPath& path, uint64_t now) const {
    const SdmaSlot* head = nullptr;
    for (int id : path.slots) {
      const SdmaSlot& s = slots_[id];
      if (engine_op(s) && (!head || s.t_submit < head->t_submit)) head = &s;
    }
    if (!head) return false;
    const uint64_t npaths = std::max<size_t>(1, n_pull_paths_) + (cu_enabled() && !cu_paused_ ? 1 : 0);
    const uint64_t since = std::max(path.t_head, head->t_submit);
    // the other direction's commands that were on this engine when the head
    // command was submitted may run first
    const uint64_t bytes = head->op_bytes + head->ahead;
    const uint64_t gbs = cfg_.overdue_gbs ? cfg_.overdue_gbs : 50;  // 1 GB/s = 1 byte per ns
    return now > since && now - since > 4 * npaths * bytes / gbs + 500000;  // ns
  }

  // The paths of this phase: the duplex paths while the other direction moves
  // (see set_peer), else the direction's own. Set at the top of every round of
  // the engine loop, before any path pulls.
  void phase(uint64_t now) {
    usable_ = peer_moving(now) ? cfg_.duplex[dir_] : cfg_.mask[dir_];
    n_pull_paths_ = 0;
    for (auto& path : paths_) n_pull_paths_ += (usable_ >> path.engine) & 1u;
    cu_paused_ = cu_enabled() && !(usable_ & MMA_PATH_CU) && n_pull_paths_ > 0;
  }
  // The same decision for the CU path alone, from any thread (paths_ and cfg_
  // are fixed after init).
  bool cu_paused_at(uint64_t now) const {
    if (!cu_enabled() || !peer_moving(now) || (cfg_.duplex[dir_] & MMA_PATH_CU)) return false;
    for (auto& path : paths_)
      if ((cfg_.duplex[dir_] >> path.engine) & 1u) return true;
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
    const uint32_t usable = usable_;
    for (size_t k = 0; k < paths_.size(); ++k) {
      SdmaPath& path = paths_[(k + rr_) % paths_.size()];
      if (!((usable >> path.engine) & 1u)) continue;  // not a path of this phase
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
          free_mask = be_->engines_idle(dir_);
          have_mask = true;
        }
        // busy with work of the other direction of this library: not foreign
        if (!(free_mask & (1u << path.engine)) && peer_bytes_on(path.engine) == 0) {
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
        const size_t share = fair_share(x, path);
        if (share == 0) break;
        const Task& t = x->tasks[i];
        const size_t end = merge_run(x, i, std::min<size_t>(cfg_.merge, share));
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
          ok = sdma_copy(s, reinterpret_cast<void*>(t.dst_dma), h2d, reinterpret_cast<void*>(t.src_dma), !h2d,
                         s.count);
          s.state = kCopy;
        } else if (x->kind == Kind::kKvFetch) {
          ok = sdma_copy(s, reinterpret_cast<void*>(s.staging), true, reinterpret_cast<void*>(t.host_dma), false,
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
          requeue_cu(x, i, end);
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
    if (x->unlaunched.load(std::memory_order_acquire) && !x->aborting) {
      x->aborting = true;  // drain what the copy engines hold; nothing else will run
      x->failed = true;
      return true;
    }
    if (!x->started && !x->ignored && (x->early || ld_acq(&r->h.started) == x->seq)) {
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
    for (uint64_t t = x->pushed; t < x->pushed + x->waves; ++t) {
      CuEntry* e = &x->ring[t % kRingSize];
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

  // How long the engine thread may sleep before its next round (Section 5.3,
  // CPU overhead): 0 to poll on. A nap must delay neither a path's next
  // micro-task nor a transfer's completion. With R the link rate the overdue
  // rule assumes, it is bounded by:
  //  - each copy engine with commands of ours in flight: half the time until
  //    the last of them could end at the fastest rate the engine may run --
  //    1.5 times its measured rate, at most R -- counted from when the first
  //    reached the head of the queue, and kLateNapNs once that time is near
  //    or past; so the thread looks often when they land and when the engine
  //    needs its next command. An engine idle while a staging step of its own
  //    runs (its next command waits for the CU side): kLateNapNs;
  //  - a transfer waiting for its start signal: a 256th of its bytes at R
  //    (the copy engines join at most that late; the CU path starts with the
  //    kernel, from its prefilled entries);
  //  - a started transfer: a 64th, at R, of its bytes that are neither landed
  //    nor in a copy-engine command, so naps shrink to nothing as the CU path
  //    finishes it, and stop once copy-engine commands hold all that is left;
  //  - its CU path, while micro-tasks remain that the CU path may take: half
  //    the time its outstanding ring entries beyond one per wave (which may
  //    be nearly done) take at R; with no more entries than that, kLateNapNs
  //    if the CU path is full (it takes nothing until a micro-task lands),
  //    else none.
  // Nor does the thread nap with a transfer submitted but not yet taken in, a
  // transfer completed or failed but not retired, or a staging step waiting
  // for ring room.
  uint64_t nap() const {
    if (!cfg_.nap_ns || n_incoming_.load(std::memory_order_relaxed)) return 0;
    const uint64_t gbs = cfg_.overdue_gbs ? cfg_.overdue_gbs : 50;  // 1 GB/s = 1 byte per ns
    const uint64_t now = now_ns();
    uint64_t ns = cfg_.nap_ns;
    // payload bytes in copy-engine commands, per transfer (few are active)
    auto& on_engines = nap_scratch_;
    on_engines.clear();
    for (const auto& path : paths_) {
      const SdmaSlot* q[64];
      size_t n = 0;
      bool staging = false;
      for (int id : path.slots) {
        const SdmaSlot& sl = slots_[id];
        if (sl.state == kH2DScatterPush || sl.state == kD2HGatherPush) return 0;
        if (engine_op(sl)) {
          if (n < 64) q[n++] = &sl;  // a path has at most queue_depth (<= 16) slots
        } else if (sl.state != kFree) {
          staging = true;
        }
      }
      if (!n) {
        if (staging) ns = std::min(ns, kLateNapNs);  // idle until a staging step of its own lands
        continue;
      }
      std::sort(q, q + n, [](const SdmaSlot* a, const SdmaSlot* b) { return a->t_submit < b->t_submit; });
      const double fast = std::max(path.ns_per_byte / 1.5, 1.0 / static_cast<double>(gbs));
      double end = static_cast<double>(std::max(path.t_head, q[0]->t_submit));
      for (size_t k = 0; k < n; ++k) {
        end += fast * static_cast<double>(q[k]->op_bytes);
        const Transfer* x = q[k]->x;
        const uint64_t b = x->kind == Kind::kLinear ? q[k]->count : q[k]->count * x->piece;
        auto it = std::find_if(on_engines.begin(), on_engines.end(), [x](const auto& e) { return e.first == x; });
        if (it == on_engines.end())
          on_engines.push_back({x, b});
        else
          it->second += b;
      }
      ns = std::min(ns, end > static_cast<double>(now + 2 * kLateNapNs)
                            ? static_cast<uint64_t>((end - static_cast<double>(now)) / 2)
                            : kLateNapNs);
    }
    for (const auto& up : active_) {
      const Transfer* x = up.get();
      if (x->completed || x->failed || x->ignored || x->aborting || x->unlaunched.load(std::memory_order_relaxed))
        return 0;
      if (!x->started) {
        ns = std::min(ns, x->bytes / gbs / 256);
        continue;
      }
      uint64_t eng = 0;
      for (const auto& e : on_engines)
        if (e.first == x) eng = e.second;
      ns = std::min(ns, (x->bytes - std::min(x->bytes, x->done_bytes + eng)) / gbs / 64);
      const bool cu_takes = (cu_enabled() && !cu_paused_) || x->pool_dev || x->cu_only_left > 0;
      if (cu_takes && x->n_claimed < x->tasks.size()) {
        if (x->cu_entries <= x->waves) {
          // Full, the CU path takes nothing more until one of its micro-tasks lands.
          if (x->cu_busy < (x->pool_dev ? 2 * x->waves : cfg_.cu_depth)) return 0;
          ns = std::min(ns, kLateNapNs);
          continue;
        }
        const uint64_t per_entry = x->kind == Kind::kLinear ? x->sub
                                   : (x->kv_per ? x->kv_per : std::max<uint64_t>(1, cfg_.sub / x->piece)) * x->piece;
        ns = std::min(ns, (x->cu_entries - x->waves) * per_entry / gbs / 2);
      }
    }
    return ns;
  }

  bool retire_ready(Transfer* x) {
    // A self-contained kernel's done tags are its last accesses to the record.
    if (x->self_contained) return x->n_done == x->tasks.size();
    if (x->unlaunched.load(std::memory_order_acquire)) return x->sdma_refs == 0;
    if (ld_acq(&x->rec->h.released) != x->seq) return false;
    // Every wave wrote its done tags before the last one released the record,
    // but `complete` may have been published before this thread saw them (the
    // early completion once only CU entries remain): credit them now, so that
    // per-path accounting is exact. Tags still missing after a grace period
    // mean a broken protocol; the transfer is then reported as failed.
    scan_cu(x);
    if (x->n_done != x->tasks.size() && !x->failed) {
      const uint64_t now = now_ns();
      if (!x->t_released) x->t_released = now;
      if (now - x->t_released < kTagGraceNs) return false;
      x->failed = true;
    }
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
          engine_waiting_ = true;
          cv_.wait_for(lk, std::chrono::milliseconds(100));
          engine_waiting_ = false;
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
      phase(now_ns());
      bool p = false;
      for (auto& up : active_) {
        up->progress = false;
        p |= advance(up.get());
        p |= scan_cu(up.get());
      }
      p |= poll_sdma();
      for (auto& up : active_) p |= pull_cu(up.get(), cu_paused_);
      p |= pull_sdma();
      for (auto& up : active_) {
        p |= advance(up.get());
        if (up->progress && !up->ignored && up->rec) st_rel(&up->rec->h.heartbeat, ++up->heartbeat);
      }
      // Retire transfers whose kernel has left the record.
      for (size_t i = 0; i < active_.size();) {
        Transfer* x = active_[i].get();
        if (!retire_ready(x)) {
          ++i;
          continue;
        }
        // A failed launch was reported to the caller; it leaves no sticky error.
        const bool unlaunched = x->unlaunched.load(std::memory_order_relaxed);
        const bool bad =
            !unlaunched && (x->failed || x->ignored || (x->rec && ld_acq(&x->rec->h.status) != 0));
        finish(x, bad, !unlaunched);
        active_.erase(active_.begin() + static_cast<long>(i));
        p = true;
      }
      bool moving = false;
      for (auto& up : active_) moving |= up->started && !up->completed && !up->failed;
      if (moving)
        moving_until_.store(now_ns() + (cfg_.duplex_hold_ns ? cfg_.duplex_hold_ns : kDuplexHoldNs),
                            std::memory_order_relaxed);
      const uint64_t nap_ns = active_.empty() ? 0 : nap();
      if (nap_ns >= kMinNapNs) {
        // A submission wakes the thread (engine_waiting_), as in the idle wait.
        idle_spins = 0;
        std::unique_lock<std::mutex> lk(mu_);
        if (incoming_.empty() && !stop_) {
          st_->naps += 1;
          engine_waiting_ = true;
          cv_.wait_for(lk, std::chrono::nanoseconds(nap_ns));
          engine_waiting_ = false;
        }
      } else if (p) {
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
  Backend* be_;
  Stats* st_;
  Record* recs_ = nullptr;
  Record* recs_dev_ = nullptr;
  uint64_t* light_ = nullptr;      // light slots' done tags, kPrefill per slot (host address)
  uint64_t* light_dev_ = nullptr;  // the same, device address
  std::unique_ptr<CuEntry[]> light_ring_;  // scratch ring: light transfers' entries go to the kernel args
  uint64_t* pool_tab_ = nullptr;      // HBM pool launches' table arena (host address)
  uint64_t* pool_tab_dev_ = nullptr;  // the same, device address
  uint32_t* pool_ctr_ = nullptr;      // per light slot: finished workgroups of its pool launch (device)
  std::vector<uint8_t> seg_used_;     // arena segments in use (mu_)
  DevState* ds_ = nullptr;
  std::vector<SdmaSlot> slots_;
  std::vector<SdmaPath> paths_;
  uint64_t stage_bytes_ = 0;
  size_t rr_ = 0;
  std::mutex mu_;
  std::condition_variable cv_, cv_done_;
  std::deque<std::unique_ptr<Transfer>> incoming_;
  std::vector<std::unique_ptr<Transfer>> active_;  // engine thread only
  std::deque<uint32_t> free_recs_, free_light_;
  // Device control: per record, the copy engines' polled completion signal and
  // its device-visible value. Transfers tracked by the submitting threads (see
  // track) that are launched and not yet retired.
  std::vector<uint64_t> dev_sig_;
  std::vector<const int64_t*> dev_sig_val_;
  std::mutex dev_mu_;  // taken before mu_, never after it
  std::deque<std::unique_ptr<Transfer>> tracked_;
  std::atomic<uint64_t> n_tracked_{0};
  uint64_t inflight_ = 0;
  // Bytes of this engine's commands in flight per copy engine; read by the
  // other direction's engine thread.
  std::atomic<uint64_t> eng_bytes_[MMA_MAX_SDMA] = {};
  std::atomic<uint64_t> moving_until_{0};  // see peer_moving (read by the other direction)
  uint32_t usable_ = 0;                    // paths of this phase (see phase)
  mutable std::vector<std::pair<const Transfer*, uint64_t>> nap_scratch_;  // see nap (engine thread)
  bool cu_paused_ = false;                 // the CU path takes only CU-only micro-tasks (see set_peer)
  size_t n_pull_paths_ = 0;                // copy-engine paths pull_sdma may use this round
  const Engine* peer_ = nullptr;          // the other direction's engine
  bool stop_ = false;
  bool engine_waiting_ = false;  // the engine thread waits on cv_ (guarded by mu_)
  std::atomic<bool> stop_flag_{false};
  std::atomic<uint64_t> n_incoming_{0};
  static constexpr uint64_t kIdleSpinNs = 2000000;  // 2 ms
  // A direction counts as moving this long after its last started transfer
  // that was not complete, so that the gaps between back-to-back transfers (a
  // weight list in groups with kernels between them) do not switch the other
  // direction's paths back and forth.
  static constexpr uint64_t kDuplexHoldNs = 1000000;  // 1 ms
  static constexpr uint64_t kTagGraceNs = 100000000;  // 100 ms
  static constexpr uint64_t kMinNapNs = 4000;  // shorter naps cost more than the polls they save
  static constexpr uint64_t kRateMinBytes = 256 * 1024;  // commands that time an engine's rate
  static constexpr uint64_t kLateNapNs = 10000;  // nap once a copy engine's commands may have landed
  static constexpr size_t kReapWindow = 512;
  std::thread thread_;
};

// Micro-tasks of a tensor list (Section 3.4 Task Manager). sizes[i] is tensor
// i's byte count; src_cu/dst_cu are the addresses the CU path uses for it.
inline std::unique_ptr<Transfer> make_list_transfer(int dir, const mma_copy_desc_t* list, uint64_t n,
                                                    const uint64_t* sizes, const uint64_t* src_cu,
                                                    const uint64_t* dst_cu, const Config& c) {
  std::vector<PlanItem> plan;
  plan_list(sizes, n, c.chunk, c.fallback, c.small, plan);
  std::unique_ptr<Transfer> x(new Transfer);  // owner/tdone are written before they are read
  x->dir = dir;
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
  return x;
}

// Micro-tasks of a block-table KV transfer: host slot host_slots[i] <-> GPU
// block gpu_blocks[i], ppb pieces of `piece` bytes per block. `host` is the
// pool's address for the copy engines, pool_cu the CU path's.
inline std::unique_ptr<Transfer> make_kv_transfer(int dir, uint64_t piece, uint32_t ppb, uint64_t host,
                                                  uint64_t pool_cu, bool pool_dev, bool sdma_ok,
                                                  const int32_t* host_slots, const int32_t* gpu_blocks, uint64_t n,
                                                  const Config& c) {
  std::vector<PlanItem> plan;
  plan_kv(n, ppb, piece, c.chunk, plan);
  std::unique_ptr<Transfer> x(new Transfer);  // owner/tdone are written before they are read
  x->dir = dir;
  x->kind = dir == MMA_H2D ? Kind::kKvFetch : Kind::kKvOffload;
  x->piece = piece;
  x->pool_dev = pool_dev;
  x->sdma_ok = sdma_ok;
  if (pool_dev) {
    x->pool_base = host;
    x->pool_pairs.resize(n);
    for (uint64_t i = 0; i < n; ++i)
      x->pool_pairs[i] = static_cast<uint32_t>(host_slots[i]) | static_cast<uint64_t>(gpu_blocks[i]) << 32;
  }
  x->tasks.reserve(plan.size());
  const uint64_t slot_bytes = piece * ppb;
  for (const PlanItem& p : plan) {
    Task t{};
    const uint64_t off = static_cast<uint64_t>(host_slots[p.item]) * slot_bytes + p.offset * piece;
    t.host_dma = host + off;
    t.host_cu = pool_cu + off;
    t.blk = static_cast<uint64_t>(gpu_blocks[p.item]);
    t.p0 = static_cast<uint32_t>(p.offset);
    t.bytes = p.bytes;
    t.flags = sdma_ok ? 0u : kPlanCuOnly;
    x->tasks.push_back(t);
  }
  return x;
}


}  // namespace mma

#endif  // MMA_ENGINE_H_
