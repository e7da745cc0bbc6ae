/*
 * mma.h -- Multipath Memory Access on one MI355X (gfx950): C ABI.
 *
 * One host<->GPU copy, tensor list or block-table KV transfer is split into
 * micro-transfers that are driven concurrently over every path the GPU owns:
 * its SDMA copy engines (submitted by a host engine thread) and CU-issued
 * zero-copy loads/stores to pinned host memory (executed by the workgroups of
 * a per-transfer "dummy-task" kernel). Paths pull work through per-path
 * outstanding queues (backpressure, no link-state feedback); completion is
 * aggregated through counters in device-visible memory, and the dummy-task
 * kernel holds the caller's stream until every fragment has landed, so
 * stream ordering is exactly that of the native copy it replaces.
 *
 * Paper: "Multipath Memory Access: Breaking Host--GPU Bandwidth Bottlenecks in
 * LLM Serving" (arXiv 2512.16056). Section numbers below refer to it. The
 * relay paths through peer GPUs (Section 3.4 relay scheduling, dual-pipeline
 * relay) need a second GPU and are not part of this library.
 *
 * Conventions for every call:
 *   - Returns mma_status_t: MMA_OK (0) or a negative error code. No call
 *     aborts the process or lets a C++ exception out (host memory exhaustion
 *     is MMA_ERR_NO_MEMORY); details of the last error: mma_last_error().
 *   - Argument validation happens before anything is enqueued: a call that
 *     fails validation has no effect.
 *   - bytes == 0 / n == 0 is an MMA_OK no-op (nothing is enqueued).
 *   - `stream` is a hipStream_t (NULL = the device's null stream) of the
 *     device passed to mma_init.
 *   - Host buffers must be pinned and device-mapped (mma_host_alloc,
 *     hipHostMalloc, or hipHostRegister with the mapped flag); pageable host
 *     memory is rejected with MMA_ERR_NOT_PINNED. Device buffers must be
 *     device memory of the initialised device.
 *   - Descriptor arrays and block tables are copied before the call returns;
 *     data buffers are borrowed until the stream has passed the transfer, as
 *     with hipMemcpyAsync.
 *   - Thread-safe: submissions are serialised internally.
 *   - Asynchronous failures (an SDMA error, a wait-kernel watchdog timeout)
 *     never hang the stream: the dummy-task kernel still exits, and every
 *     later call returns the sticky MMA_ERR_TRANSFER_FAILED until
 *     mma_clear_error().
 */
#ifndef MMA_H_
#define MMA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t mma_status_t;

#define MMA_OK 0
#define MMA_ERR_NOT_INITIALIZED (-1)
#define MMA_ERR_INVALID_ARG (-2)
#define MMA_ERR_NOT_PINNED (-3)
#define MMA_ERR_HIP (-4)
#define MMA_ERR_HSA (-5)
#define MMA_ERR_TRANSFER_FAILED (-6)
#define MMA_ERR_ALREADY_INITIALIZED (-7)
#define MMA_ERR_NO_MEMORY (-8)
#define MMA_ERR_BUFFER_TOO_SMALL (-9)
#define MMA_ERR_TIMEOUT (-10)
#define MMA_ERR_INTERNAL (-11) /* a C++ exception inside the library other than host memory
                                  exhaustion (MMA_ERR_NO_MEMORY); mma_last_error() names it */

/* Direction of a transfer. Only host<->device copies are handled (Section 3.2:
 * GPU-to-GPU traffic is not intercepted). */
#define MMA_H2D 0
#define MMA_D2H 1

/* Path mask bits: bit e (e < 16) = SDMA engine e; MMA_PATH_CU = the CU path. */
#define MMA_PATH_CU 0x80000000u
/* duplex_paths_*: keep a direction's own paths while the other direction moves. */
#define MMA_DUPLEX_UNCHANGED 0xFFFFFFFFu
#define MMA_MAX_SDMA 16
#define MMA_NUM_PATHS 17      /* stats index 16 = CU path */
#define MMA_MAX_LAYERS 256    /* KV layers per call */

/* Runtime tunables (Section 4, deployment: chunk size, thresholds and path
 * set are configuration). Zero in any field selects its default. */
typedef struct mma_config {
  uint64_t chunk_bytes;     /* micro-task size; default 2 MiB (Section 3.4 Task Manager, 5.3) */
  uint64_t fallback_bytes;  /* requests (or list tensors) below this are a single micro-task;
                               default 2 * chunk_bytes (Section 3.2 fallback, 5.3 threshold) */
  uint64_t small_bytes;     /* tensors below this are CU-path-only; default 64 KiB */
  uint32_t queue_depth;     /* outstanding micro-tasks per SDMA engine; default 2 (Section 5.3) */
  uint32_t cu_queue_depth;  /* outstanding micro-tasks on the CU path; default 4 */
  uint32_t backoff_depth;   /* once a path's queue is full it pulls again only when its depth
                               drops below this (Section 3.4 contention back-off);
                               default: each path's own queue depth (no extra back-off);
                               a value given applies to every path */
  uint32_t path_mask_h2d;   /* paths used host->device; default: CU path + the host-facing
                               SDMA engines reported by ROCr */
  uint32_t path_mask_d2h;   /* paths used device->host; same default */
  uint32_t cu_workgroups;   /* max workgroups (4 wave64 each) of the dummy-task kernel; default 16,
                               at most 256 (x-packed KV transfers use up to 1.5 times this:
                               their waves spend part of their time writing out an LDS tile);
                               chunk_bytes / cu_sub_bytes must not exceed 2048 */
  uint32_t cu_sub_bytes;    /* bytes one wave moves per CU claim; default 64 KiB */
  uint32_t watchdog_ms;     /* wait-kernel gives up after this long without engine progress;
                               default 20000 */
  uint32_t static_split;    /* 0 (default): pull-based path selection. 1: the baseline the paper
                               compares against (Section 5.1.2) -- a fixed split decided at plan
                               time: static_cu_percent of the micro-tasks (interleaved) go to the
                               CU path, the rest to the SDMA engines (which share them by pulling) */
  uint32_t static_cu_percent; /* also, under MMA_CONTROL_DEVICE, the CU path's share of a linear
                               transfer's bytes when the copy engines take part (0: 40) */
  uint32_t sdma_merge_tasks; /* at most this many micro-tasks that follow each other in both
                               address spaces (a linear run, or one KV block's consecutive pieces)
                               go to an SDMA engine as one command, and never more than the
                               engine's fair share of the transfer's remaining work; default:
                               64 MiB worth (max(1, 64 MiB / chunk_bytes)); 1 = one command per
                               micro-task */
  uint32_t cu_whole_bytes;  /* host->device: a copy or tensor list of at most this many bytes,
                               whose micro-tasks fit one launch (at most 48 CU entries), is carried
                               by the CU path alone in a dummy-task launch that needs no host round
                               trip (no start signal, no completion wait) -- below this size the
                               setup of several paths costs more than it gains (Section 3.2
                               fallback); default 24 MiB; 1 keeps every transfer on the multipath
                               engine */
  uint32_t cu_whole_bytes_d2h; /* the same for device->host; default 8 MiB (CU stores to host
                               memory reach the link less efficiently than CU loads, measured) */
  uint32_t control;         /* who drives a transfer once it is submitted (Section 6, Current
                               limitations: a CPU-driven control plane costs fine-grained
                               transfers scheduling time):
                               MMA_CONTROL_HOST (0, default): the engine thread of the direction
                                 pulls micro-tasks for every path while the transfer runs;
                               MMA_CONTROL_DEVICE (1): the calling thread plans the whole transfer
                                 at submission -- every CU-path entry is published before the
                                 launch, and on a stream with nothing pending the copy engines get
                                 a fixed share of a linear transfer at once -- and the dummy-task
                                 kernel alone tracks completion; no host thread works on the
                                 transfer afterwards (records are recycled by later calls). On a
                                 stream with work pending, and for KV transfers, the CU path
                                 carries the transfer alone. A copy or tensor list of more than
                                 4096 micro-tasks is planned again at twice chunk_bytes until it
                                 fits; a KV transfer of more goes to the engine thread. */
  uint32_t duplex_paths_h2d; /* paths host->device pulls from while a device->host transfer is
                               moving (Section 5.1.2, concurrent flows; host control only).
                               0 (default): the SDMA engines of path_mask_h2d, without the CU
                               path. MMA_DUPLEX_UNCHANGED: path_mask_h2d. Each copy engine
                               runs one in-order queue for both directions, and CU zero-copy loads
                               send their read requests up the lanes that device->host data uses.
                               Micro-tasks only the CU path may carry still take it. */
  uint32_t duplex_paths_d2h; /* paths device->host pulls from while a host->device transfer is
                               moving. 0 (default): with the default path_mask_d2h, SDMA engines
                               2-5 (on MI355X the xGMI-facing engines, 13-18 GB/s each toward the
                               host), neither the host-facing engines nor the CU path, whose stores
                               to host memory share the upstream lanes in small writes; with a
                               path_mask_d2h given, its SDMA engines without the CU path.
                               MMA_DUPLEX_UNCHANGED: path_mask_d2h.
                               Engines the device does not offer are dropped; a set left with no
                               path, or a CU path the direction does not have, falls back to its
                               path mask. */
  uint32_t engine_nap_us;   /* host control: the longest a direction's engine thread sleeps between
                               two rounds of its loop (Section 5.3, CPU overhead). It sleeps only
                               while every path has work queued for longer than the nap and no
                               transfer is near its end, and a submission wakes it at once.
                               Default 50; MMA_ENGINE_NAP_OFF: poll without sleeping while a
                               transfer is in flight (the paper's engine); at most 1000. */
} mma_config_t;
#define MMA_ENGINE_NAP_OFF 0xFFFFFFFFu

typedef struct mma_copy_desc {
  void* dst;
  const void* src;
  uint64_t bytes;
} mma_copy_desc_t;

/* Paged KV layout (Section 2.1 KV offload/fetch; the layouts themselves are
 * readings, the paper does not state them):
 *   piece     = block_tokens * kv_heads * head_dim * elem_bytes bytes: one layer's
 *               K or V of one block, token-major [block_tokens][kv_heads][head_dim]
 *               in host memory;
 *   host pool = host_num_slots slots, slot s = [num_layers][2 (K,V)][piece];
 *   GPU layer l (one pointer per layer) = [2 (K,V)][gpu_num_blocks][block], where a
 *               block holds one piece in the GPU block layout `gpu_layout`:
 *     MMA_KV_LAYOUT_PIECE   (0): as in host memory;
 *     MMA_KV_LAYOUT_XPACKED (1): the layout of paged-attention decode kernels --
 *               key [kv_heads][head_dim / x][block_tokens][x] with x = 16 / elem_bytes,
 *               value [kv_heads][head_dim][block_tokens]. Needs elem_bytes in
 *               {1, 2, 4, 8}, head_dim * elem_bytes and block_tokens * elem_bytes
 *               multiples of 16, a 16-byte-aligned pool and layer tensors, and
 *               block_tokens * (head_dim * elem_bytes + 16) <= 36 KiB (one head of
 *               one block fits a wave's LDS tile); otherwise MMA_ERR_INVALID_ARG.
 *     MMA_KV_LAYOUT_HND     (2): head-major, K and V alike [kv_heads][block_tokens][head_dim]
 *               (the transposed layout of some attention kernels). Needs
 *               head_dim * elem_bytes a multiple of 16 and a 16-byte-aligned pool and
 *               layer tensors; otherwise MMA_ERR_INVALID_ARG. */
#define MMA_CONTROL_HOST 0u
#define MMA_CONTROL_DEVICE 1u

#define MMA_KV_LAYOUT_PIECE 0u
#define MMA_KV_LAYOUT_XPACKED 1u
#define MMA_KV_LAYOUT_HND 2u
typedef struct mma_kv_layout {
  uint32_t num_layers;
  uint32_t block_tokens;
  uint32_t kv_heads;
  uint32_t head_dim;
  uint32_t elem_bytes;
  uint32_t gpu_num_blocks;
  uint32_t host_num_slots;
  uint32_t gpu_layout;    /* MMA_KV_LAYOUT_PIECE (0), MMA_KV_LAYOUT_XPACKED (1) or MMA_KV_LAYOUT_HND (2) */
} mma_kv_layout_t;

typedef struct mma_stats {
  uint64_t transfers;                     /* transfers retired */
  uint64_t failed_transfers;
  uint64_t path_bytes[MMA_NUM_PATHS];     /* payload bytes carried per path */
  uint64_t path_tasks[MMA_NUM_PATHS];     /* micro-tasks carried per path */
  uint64_t staging_bytes;                 /* HBM<->HBM bytes moved through SDMA staging */
  uint64_t sdma_submit_failures;          /* submissions re-routed to the CU path */
  uint64_t engine_cpu_ns;                 /* CPU time consumed by the engine threads */
  uint64_t engine_wall_busy_ns;           /* wall time with at least one transfer active */
  uint64_t sdma_foreign_busy_skips;       /* pulls skipped: engine busy with another component's copies */
  uint64_t sdma_congestion_backoffs;      /* engines backed off after an overdue command */
  uint64_t sdma_commands;                 /* copy-engine commands issued (a command may carry several
                                             adjacent micro-tasks) */
  uint32_t sdma_engines_h2d;              /* masks actually in use */
  uint32_t sdma_engines_d2h;
  uint32_t cu_path_enabled;
  uint32_t reserved;
  uint64_t pool_launches;                 /* KV transfers with the pool in this GPU's memory carried by
                                             one pool-kernel launch (the others took the ring path) */
  uint64_t engine_naps;                   /* sleeps of the engine threads between rounds of their loop
                                             while transfers were in flight (engine_nap_us) */
} mma_stats_t;

/* One micro-task of a plan (host-only planner, exposed for verification).
 * Linear/list plans: item = tensor index, offset = byte offset in the tensor,
 * bytes = length, flags bit 0 = CU-path-only.
 * KV plans: item = table index i, offset = first piece (2*l + k), bytes = piece count. */
typedef struct mma_plan_entry {
  uint64_t item;
  uint64_t offset;
  uint64_t bytes;
  uint32_t flags;
  uint32_t reserved;
} mma_plan_entry_t;

#define MMA_TASK_CU_ONLY 1u
#define MMA_TASK_SDMA_ONLY 2u

/* ---------------------------------------------------------------- lifecycle */

/* Fill *out with the built-in defaults (no environment overrides, no GPU needed). */
mma_status_t mma_config_default(mma_config_t* out);

/* Initialise the library on HIP device `hip_device`: map it to its ROCr agent,
 * discover its SDMA engines, allocate transfer records, and start one engine
 * thread per direction (Section 4, Multipath Transfer Engine: separate H2D and
 * D2H engines). cfg == NULL: defaults, then MMA_* environment overrides
 * (MMA_CHUNK_BYTES, MMA_FALLBACK_BYTES, MMA_SMALL_BYTES, MMA_QUEUE_DEPTH,
 * MMA_CU_QUEUE_DEPTH, MMA_BACKOFF_DEPTH, MMA_PATHS_H2D, MMA_PATHS_D2H,
 * MMA_CU_WGS, MMA_CU_SUB_BYTES, MMA_WATCHDOG_MS, MMA_SDMA_MERGE_TASKS,
 * MMA_CU_WHOLE_BYTES, MMA_CU_WHOLE_BYTES_D2H, MMA_CONTROL, MMA_STATIC_CU_PERCENT,
 * MMA_DUPLEX_PATHS_H2D, MMA_DUPLEX_PATHS_D2H, MMA_ENGINE_NAP_US, MMA_TRACE).
 * As in cfg, 0 selects a field's default; an environment value that does not
 * parse as a number reads as 0. Errors: MMA_ERR_ALREADY_INITIALIZED, MMA_ERR_INVALID_ARG (bad device or
 * config), MMA_ERR_HIP / MMA_ERR_HSA. */
mma_status_t mma_init(int hip_device, const mma_config_t* cfg);

/* Wait for every submitted transfer to retire (bounded), stop the engine
 * threads and release library resources. Returns MMA_ERR_TIMEOUT if in-flight
 * transfers did not drain (their streams are then still blocked). Must not run
 * concurrently with other calls of this library. A process that exits without
 * it has its engine threads stopped when the library is unloaded, before the
 * HIP runtime's own teardown. */
mma_status_t mma_finalize(void);

/* The configuration in effect (after defaults and environment). */
mma_status_t mma_get_config(mma_config_t* out);

/* Host-side wait until every transfer submitted so far has retired, or
 * timeout_ms elapsed (MMA_ERR_TIMEOUT). Does not synchronise any stream.
 * Retired means that no path of the library touches the transfer's buffers
 * any more. Device-to-host data is then in host memory (every wave releases
 * at system scope before its done tag). Data written to this GPU's memory is
 * ordered for later work by the transfer's stream, as for any copy or kernel:
 * work on another stream must wait for that stream (an event) -- a retired
 * transfer does not make it visible there, in particular not a KV transfer
 * with its pool in this GPU's memory, whose workgroups release nothing when
 * they finish (a device-wide release per workgroup costs HBM bandwidth). */
mma_status_t mma_synchronize(uint32_t timeout_ms);

/* ------------------------------------------------------------ host memory */

/* Pinned, device-mapped host memory, allocated on the GPU-local NUMA node when
 * the platform reports one (Section 5.1 methodology: pinned host buffers).
 * *out receives a pointer usable both by the host and as a kernel argument.
 * Owned by the caller; free with mma_host_free. bytes == 0 -> *out = NULL. */
mma_status_t mma_host_alloc(uint64_t bytes, void** out);
mma_status_t mma_host_free(void* p);

/* ---------------------------------------------------------------- transfers */

/* Asynchronous copy of `bytes` bytes with hipMemcpyAsync semantics on `stream`
 * (Section 3.1 workflow; Section 3.2 Transfer Task Interceptor; Section 3.3
 * Sync Engine). dir = MMA_H2D: src pinned host, dst device; MMA_D2H: src
 * device, dst pinned host. The stream-visible completion happens only after
 * every micro-transfer has landed: work enqueued on `stream` after this call
 * sees the whole copy, work before it is complete before any byte is read.
 * Errors: MMA_ERR_INVALID_ARG (NULL with bytes > 0, bad dir, pointer of the
 * wrong kind for dir), MMA_ERR_NOT_PINNED, MMA_ERR_HIP (launch failure),
 * MMA_ERR_TRANSFER_FAILED (sticky), MMA_ERR_NOT_INITIALIZED. */
mma_status_t mma_memcpy_async(void* dst, const void* src, uint64_t bytes, int32_t dir, void* stream);

/* Synchronous copy with hipMemcpy semantics (Section 3.2: the blocking call
 * returns once the data has arrived). The copy is enqueued on the legacy
 * default stream, so it is ordered after earlier work there and on other
 * blocking streams; the call returns after that stream has passed it and the
 * engine has retired it, so a failure of this copy is returned here
 * (MMA_ERR_TRANSFER_FAILED). Arguments, pinning rules and other errors as for
 * mma_memcpy_async; MMA_ERR_TIMEOUT if the transfer is not retired within the
 * watchdog period plus 10 s. Equal to mma_memcpy_stream(..., NULL, NULL). */
mma_status_t mma_memcpy(void* dst, const void* src, uint64_t bytes, int32_t dir);

/* What happened to the copy of a synchronous call (mma_memcpy_stream's
 * `outcome`): NOT_ENQUEUED -- refused, or its launch failed; no part of it is
 * in flight (an MMA_ERR_TRANSFER_FAILED here is the sticky failure of an
 * earlier transfer). RETIRED -- every path has finished with it: MMA_OK, or
 * MMA_ERR_TRANSFER_FAILED if this copy failed (its destination may then hold
 * partial data, and nothing writes it any more). IN_FLIGHT -- enqueued and
 * not retired within the limit (MMA_ERR_TIMEOUT, or MMA_ERR_HIP from the
 * stream wait): parts of it may still be moving. */
#define MMA_COPY_NOT_ENQUEUED 0
#define MMA_COPY_RETIRED 1
#define MMA_COPY_IN_FLIGHT 2

/* Synchronous copy ordered on `stream`, with hipMemcpyWithStream semantics
 * (Section 3.2: a blocking copy returns once the data has arrived): enqueued on
 * `stream` like mma_memcpy_async, then the call waits until the stream has
 * passed it and the engine has retired it, so this copy's own failure is
 * returned here (MMA_ERR_TRANSFER_FAILED). If `outcome` is not NULL, it
 * receives one of MMA_COPY_* above, which tells a caller that wants to retry
 * the copy some other way whether that is safe (only when nothing of it is in
 * flight). Arguments, pinning rules and other errors as for mma_memcpy. */
mma_status_t mma_memcpy_stream(void* dst, const void* src, uint64_t bytes, int32_t dir, void* stream,
                               int32_t* outcome);

/* One logical transfer of a list of n independent copies, e.g. all weight
 * tensors of a model (Section 2.1 model wake-up; Section 5.2.2). One dummy
 * task covers the whole list. Each tensor is chunked on its own; tensors below
 * small_bytes are CU-path-only. All copies share `dir`. Destination ranges
 * must be pairwise disjoint (MMA_ERR_INVALID_ARG otherwise). `list` is copied
 * before return. */
mma_status_t mma_weights_load(const mma_copy_desc_t* list, uint64_t n, int32_t dir, void* stream);

/* KV fetch, host pool -> paged GPU cache (Section 2.1 "fetching cached KV
 * pages"; Section 5.2.1). For every i < n_blocks, l < num_layers, k in {K,V}:
 *   gpu_layers[l][k][gpu_blocks[i]] = host_pool[host_slots[i]][l][k]
 * Other GPU blocks are untouched. gpu_layers: num_layers device pointers, each
 * to [2][gpu_num_blocks][piece]; host_pool: host_num_slots slots of pinned host
 * memory -- or of device memory of this GPU (an HBM-resident KV tier), in which
 * case the transfer is an HBM gather carried by the CU path alone.
 * Tables: int32, host_slots[i] in [0, host_num_slots), gpu_blocks[i] in
 * [0, gpu_num_blocks), gpu_blocks distinct (MMA_ERR_INVALID_ARG otherwise).
 * The pointer array and both tables are copied before return. */
mma_status_t mma_kv_fetch(const mma_kv_layout_t* layout, const void* host_pool, void* const* gpu_layers,
                          const int32_t* host_slots, const int32_t* gpu_blocks, uint64_t n_blocks,
                          void* stream);

/* KV offload, paged GPU cache -> host pool (Section 2.1 offload). For every
 * j < n_blocks, l, k:  host_pool[host_slots[j]][l][k] = gpu_layers[l][k][gpu_blocks[j]].
 * Other host slots are untouched. host_slots distinct; ranges as for fetch; the
 * pool may likewise be device memory (HBM scatter, CU path only).
 * Producer work enqueued on `stream` before this call is complete and visible
 * before any byte is read. */
mma_status_t mma_kv_offload(const mma_kv_layout_t* layout, void* host_pool, const void* const* gpu_layers,
                            const int32_t* gpu_blocks, const int32_t* host_slots, uint64_t n_blocks,
                            void* stream);

/* KV fetch that allocates nothing, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc. The same operation, arguments, validation and errors as
 * mma_kv_fetch (every GPU block layout; a pinned host pool or a pool in this
 * GPU's memory), and the same bytes in the GPU cache. It makes no hipMalloc,
 * hipHostMalloc or hipFree call and uses no buffer of the engine: the block
 * table and a claim counter live in `scratch`, a fixed array of the library's
 * device code (256 B + 8 B per block, 512 KiB + 256 B in all per GPU, held
 * until the process ends), whose address mma_init looks up. The table reaches
 * it through the arguments of ceil(n_blocks / 448) small kernel launches on
 * `stream`, then one launch carries every piece on the CU path alone (no copy
 * engine, no engine thread); the transfer is complete when that launch
 * completes on the stream, and it does not appear in mma_get_stats.
 * n_blocks at most 65536: larger calls return MMA_ERR_INVALID_ARG and enqueue
 * nothing. Every call on one GPU shares its scratch array, which keeps the
 * last call's table: calls that may overlap on one GPU (other streams, other
 * threads) race and must be ordered by the caller (one stream, or events). */
mma_status_t mma_kv_fetch_noalloc(const mma_kv_layout_t* layout, const void* host_pool, void* const* gpu_layers,
                                  const int32_t* host_slots, const int32_t* gpu_blocks, uint64_t n_blocks,
                                  void* stream);

/* Dependent HBM-bound check kernel (the mixed-contention workload's consumer):
 * adds, modulo 2^64, digest = sum_i (w_i + 1) * (2i + 1) over the little-endian
 * 32-bit words w_i of dev_ptr[0, bytes) (a trailing partial word is zero-
 * padded) into *dev_out, ordered on `stream`. *dev_out is device memory the
 * caller zeroed. Verifies that loads are visible to later stream work
 * (Section 3.3 ordering requirement). */
mma_status_t mma_digest_u32(const void* dev_ptr, uint64_t bytes, uint64_t* dev_out, void* stream);

/* ------------------------------------------------------------------- status */

/* Counters since mma_init or mma_reset_stats. They cover every transfer retired so far;
 * this call first retires the transfers whose kernel has finished and that no engine
 * thread watches (whole transfers, and every transfer under MMA_CONTROL_DEVICE). */
mma_status_t mma_get_stats(mma_stats_t* out);
mma_status_t mma_reset_stats(void);
const char* mma_status_str(mma_status_t s);
/* Thread-local text of the last error reported to this thread (never NULL). */
const char* mma_last_error(void);
/* Clear the sticky asynchronous-failure state. */
mma_status_t mma_clear_error(void);

/* ------------------------------------------------- host-only (no GPU needed) */

/* The micro-task split of a tensor list (a single copy is a list of one):
 * fixed chunks from offset 0, last one shorter; a tensor below `fallback` is
 * one micro-task; below `small` it is CU-path-only (Section 3.4 Task Manager;
 * Section 3.2 fallback). Writes up to `cap` entries to out and the total
 * count to *n_out (MMA_ERR_BUFFER_TOO_SMALL if cap < total; out may then be
 * NULL to query the count). */
mma_status_t mma_plan_list(const uint64_t* sizes, uint64_t n, uint64_t chunk, uint64_t fallback,
                           uint64_t small, mma_plan_entry_t* out, uint64_t cap, uint64_t* n_out);

/* The micro-task split of a KV transfer: per table entry, consecutive pieces
 * (piece index 2*l + k) in groups of max(1, chunk / piece_bytes). */
mma_status_t mma_plan_kv(uint64_t n_blocks, uint32_t pieces_per_block, uint64_t piece_bytes, uint64_t chunk,
                         mma_plan_entry_t* out, uint64_t cap, uint64_t* n_out);

/* Byte sizes a KV layout implies (the layout described at mma_kv_layout_t): one
 * piece, one host slot (2 * num_layers pieces), the host pool (host_num_slots
 * slots) and one GPU layer tensor (2 * gpu_num_blocks pieces), i.e. what a caller
 * allocates. Any output pointer may be NULL. MMA_ERR_INVALID_ARG, and nothing
 * written, if a field is 0, num_layers > MMA_MAX_LAYERS, the piece is above
 * 4 GiB or a size does not fit 64 bits; the KV calls apply the same check. The
 * GPU block layout's own conditions are checked by the KV calls alone. */
mma_status_t mma_kv_layout_sizes(const mma_kv_layout_t* layout, uint64_t* piece_bytes, uint64_t* slot_bytes,
                                 uint64_t* pool_bytes, uint64_t* layer_bytes);

/* Block-table check applied by mma_kv_fetch/offload: equal lengths implied,
 * src[i] in [0, src_count), dst[i] in [0, dst_count), dst entries distinct.
 * MMA_OK or MMA_ERR_INVALID_ARG. */
mma_status_t mma_validate_kv_tables(const int32_t* src, uint32_t src_count, const int32_t* dst,
                                    uint32_t dst_count, uint64_t n);

/* ------------------------------------------------------------------ tracing */

/* Per-transfer timeline, recorded when a transfer retires (Section 5: transfer
 * latency and per-path load). Timestamps are CLOCK_MONOTONIC nanoseconds of the
 * host: API entry, submission (after validation and planning), first
 * observation of the start signal, first SDMA
 * submission (0 if none), last micro-task landed, `complete` published, and
 * retirement (the dummy-task kernel has left the record). kind: 0 copy/list,
 * 1 KV fetch, 2 KV offload. path_tasks: micro-tasks carried per path. */
typedef struct mma_trace_rec {
  uint64_t seq;
  int32_t dir;
  int32_t kind;
  uint64_t bytes;
  uint64_t tasks;
  uint64_t t_api_ns, t_submit_ns, t_started_ns, t_first_sdma_ns, t_last_task_ns, t_complete_ns, t_retire_ns;
  uint64_t path_tasks[MMA_NUM_PATHS];
  int32_t failed;
  int32_t reserved;
} mma_trace_rec_t;

/* Start (on != 0: the buffer is cleared) or stop recording. Also enabled by
 * MMA_TRACE=1 at mma_init. At most 65536 records are kept (oldest dropped). */
mma_status_t mma_trace_enable(int32_t on);
/* Move up to cap of the oldest records into out; *n_out = number moved. */
mma_status_t mma_trace_read(mma_trace_rec_t* out, uint64_t cap, uint64_t* n_out);

/* ------------------------------------------------------------ test hooks */

/* Faults forced from the host so that failure handling can be tested without
 * any kernel faulting or hanging: every wait stays bounded.
 *   MMA_FAULT_ENGINE_STALL_US: engine threads sleep `value` us before serving a
 *     newly started transfer (stream must stay blocked, data stays correct).
 *   MMA_FAULT_SDMA_SUBMIT_FAIL: the next `value` SDMA submissions fail; their
 *     micro-tasks are re-routed to another path.
 *   MMA_FAULT_ENGINE_IGNORE: while value != 0, engine threads do not serve newly
 *     started transfers, so the wait kernel's watchdog must release the stream.
 *   MMA_FAULT_DEVICE_SIGNAL_HOLD: under MMA_CONTROL_DEVICE, the next `value`
 *     transfers that give the copy engines a share count one command more than
 *     they submit, so the kernel's wait never sees the engines finish and its
 *     watchdog must release the stream; the count is taken back once the kernel
 *     has left, and the transfer fails (sticky).
 *   MMA_FAULT_POOL_NO_TABLE: while value != 0, a KV transfer whose pool is in
 *     this GPU's memory finds no room for its table in the pool kernel's table
 *     arena, so it takes the ring path (as when the arena is full).
 * value 0 clears a fault. */
#define MMA_FAULT_ENGINE_STALL_US 1
#define MMA_FAULT_SDMA_SUBMIT_FAIL 2
#define MMA_FAULT_ENGINE_IGNORE 3
#define MMA_FAULT_DEVICE_SIGNAL_HOLD 4
#define MMA_FAULT_POOL_NO_TABLE 5
mma_status_t mma_test_set_fault(int32_t kind, uint64_t value);

#ifdef __cplusplus
}
#endif

#endif /* MMA_H_ */
