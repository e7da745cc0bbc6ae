// Host <-> GPU protocol of one transfer: the record that the host engine thread
// and the dummy-task kernel share, and the kernel's launch arguments.
//
// A record lives in coherent (fine-grained) pinned host memory, mapped into the
// GPU's address space. Every field has exactly one writer:
//   host -> GPU : seq, closed, cu_total, complete, heartbeat, KV geometry,
//                 ring entries (payload, then tag)
//   GPU  -> host: started, released, status, done[]
// Values are epoch-stamped with the transfer's sequence number, which never
// repeats, so nothing is ever reset between uses of a record (no ABA).
//
// The CU ring is the CU path's outstanding queue (Section 3.4, Path Selector:
// one outstanding queue per path). The engine thread appends entries; waves of
// the dummy-task kernel claim them in ticket order with a device-memory atomic,
// so the GPU side needs no PCIe atomics.
#ifndef MMA_PROTO_H_
#define MMA_PROTO_H_

#include <stdint.h>

namespace mma {

constexpr uint32_t kRingSize = 4096;   // CU ring entries per record
constexpr uint32_t kRecords = 64;      // records per direction (transfers in flight)
// Light slots per direction: a transfer carried whole by one self-contained
// launch needs no record, only its done tags (at most kPrefill).
constexpr uint32_t kLightSlots = 4096;
constexpr uint32_t kMaxWorkgroups = 256;  // dummy-task kernel size limit (ring keeps one slot per wave)
constexpr uint32_t kPrefill = 48;      // ring entries also passed in the kernel arguments (linear kinds)
constexpr uint32_t kMaxLayers = 256;   // KV layer pointers per record
constexpr uint32_t kMaxLdsPerWave = 36 * 1024;  // x-packed KV tiles: 4 waves x 36 KiB + 2 KiB of a CU's 160 KiB
constexpr uint32_t kWave = 64;
constexpr uint32_t kWavesPerWG = 4;
constexpr uint32_t kBlock = kWave * kWavesPerWG;
// HBM pool launches (a paged-KV transfer whose pool is in device memory): a
// piece is moved in spans of kPoolSpan bytes, one 16-byte unit per lane and
// register, at most kPoolMaxWorkgroups workgroups per launch. The block table
// goes to the kernel through an arena of kPoolTabEntries 8-byte entries in
// device-visible host memory, handed out in segments of kPoolTabSeg entries.
constexpr uint32_t kPoolSpan = 8 * 1024;
constexpr uint32_t kPoolMaxWorkgroups = 8192;
constexpr uint32_t kPoolTabEntries = 1u << 19;
constexpr uint32_t kPoolTabSeg = 512;

// GPU block layouts of a paged-KV piece (one layer's K or V of one block). The
// host side is always token-major [tokens][heads][head_dim].
enum : uint32_t {
  kKvLayoutPiece = 0,    // the GPU block holds the piece as the host does
  kKvLayoutXPacked = 1,  // key [heads][head_dim/x][tokens][x], x = 16 / elem; value [heads][head_dim][tokens]
  kKvLayoutHnd = 2,      // head-major: K and V [heads][tokens][head_dim]
};

// Entry kinds. Kind and first piece share one 32-bit word: kind | p0 << 8.
enum : uint32_t {
  kEntryCopy = 1,       // a -> b, `count` bytes
  kEntryToPaged = 2,    // contiguous pieces at a -> GPU layers, block b, pieces p0 .. p0+count
  kEntryFromPaged = 3,  // GPU layers, block b, pieces p0 .. p0+count -> contiguous at a
  kEntryEnd = 4,        // no more work: the wave holding this ticket leaves
  kEntryKindMask = 0x7F,
  // Flag: the source was written by a copy engine while the kernel runs (SDMA
  // staging); the wave must acquire (invalidate its caches) before reading it.
  kEntryAcquire = 0x80,
};

// One cache line. The engine writes the payload, then tag0 and tag1; a wave
// reads words 0..4 with a single load instruction and accepts the entry only
// if both tags carry the expected ticket, so one PCIe read both polls for the
// entry and delivers it.
struct alignas(64) CuEntry {
  uint64_t tag0;
  uint64_t a;
  uint64_t b;
  uint32_t count;
  uint32_t kind_p0;
  uint64_t tag1;
  uint64_t pad[3];
};

struct alignas(64) RecordHdr {
  // cache line 0: host -> GPU control
  uint64_t seq;
  uint64_t closed;       // == seq: no more ring entries will be appended
  uint64_t cu_total;     // number of entries appended (valid once closed == seq)
  uint64_t complete;     // == seq: every micro-task has landed; the wait may end
  uint64_t heartbeat;    // bumped on engine progress; re-arms the kernel watchdog
  uint64_t pad0[3];
  // cache line 1: GPU -> host
  uint64_t started;      // == seq once the stream reached the dummy task
  uint64_t pad1[7];
  // cache line 2: GPU -> host
  uint64_t released;     // == seq once the kernel is done with this record
  int32_t status;        // 0 ok, 1 watchdog expired, 2 a copy-engine command failed (device control)
  int32_t pad2a;
  uint64_t pad2[6];
};

struct Record {
  RecordHdr h;
  CuEntry ring[kRingSize];
  uint64_t done[kRingSize];  // GPU -> host: tag of the entry completed in this slot
};

// Per-record scratch in device memory, shared by the waves of one kernel.
// The last wave to leave resets it before releasing the record.
struct alignas(128) DevState {
  uint64_t cursor;     // next ticket to claim
  uint32_t arrived;    // waves that have started
  uint32_t exited;     // waves that have finished claiming
  uint32_t timed_out;  // a wave's watchdog expired
  uint32_t pad[27];
};

struct KernelArgs {
  Record* rec;              // device-visible address of the record (null for a light slot)
  DevState* ds;
  uint64_t* done;           // device-visible done tags: the record's, or a light slot's kPrefill
  uint64_t seq;
  uint64_t watchdog_ticks;  // wall-clock ticks without progress before giving up
  uint32_t total_waves;
  uint32_t release_each;    // 1: system-scope release before each done flag
  // Device control (no engine thread in the loop): every CU entry is in the
  // ring before the launch, so tickets [0, n_total) are the whole CU share and
  // a ticket past it ends a wave's claims; the last wave then waits until the
  // copy engines' completion signal, whose value sdma_left points at (null if
  // they carry nothing), has counted down to 0 -- negative if a command failed.
  const int64_t* sdma_left;
  uint32_t device_ctl;
  uint32_t n_total;
  // KV geometry (unused by linear transfers)
  uint64_t kv_piece_bytes;
  uint64_t kv_kstride;      // bytes between the K and V halves of a GPU layer tensor
  uint32_t kv_layers;
  uint32_t n_pre;           // tickets [0, n_pre) are also given below: no first poll for them
  uint32_t self_contained;  // 1: the n_pre entries are the whole transfer and no copy engine takes
                            // part: wave w runs entry w and writes done[w]; a linear one is
                            // launched as mma_whole_kernel with WholeArgs instead
  // GPU block layout of paged-KV pieces: kKvLayoutPiece (as in host memory) or
  // kKvLayoutXPacked, whose geometry follows (a row is one token's head_dim
  // elements of one head: head_dim * elem bytes).
  uint32_t kv_layout;
  uint32_t kv_tokens, kv_heads, kv_row_bytes, kv_elem;
  uint32_t kv_lds_wave;     // kKvLayoutXPacked: dynamic LDS bytes per wave (the launch asks for 4x)
  // HBM pool launch (pool_tab non-null): the whole transfer is one launch of
  // mma_kv_pool_kernel, converted from these arguments (see PoolArgs).
  const uint64_t* pool_tab;  // per block: pool slot | GPU block << 32 (device-visible host memory)
  uint32_t* pool_ctr;        // device counter of finished workgroups, 0 between launches
  uint64_t pool_base;        // device address of the pool
  uint64_t pool_units;       // spans in the transfer
  uint64_t pool_per_wg;      // spans per workgroup
  uint32_t pool_spans;       // spans per piece
  uint32_t pool_to_paged;    // 1: pool -> layers (fetch); 0: layers -> pool (offload)
  uint64_t layer_ptr[kMaxLayers];
  uint64_t pre[kPrefill][3];  // words a, b, count|kind_p0 of the first ring entries
};

// Arguments of an HBM pool launch (GPU blocks in the piece or the head-major
// layout). Span u is span s of piece p of block i,
// u = (i * ppb + p) * spans + s (ppb = 2 * layers pieces per block, piece p =
// layer p / 2, K for even p and V for odd); workgroup g takes spans
// [g * per_wg, (g + 1) * per_wg). The workgroup that finishes last writes
// done[0] = make_tag(seq, 0) and returns the counter to 0.
struct PoolArgs {
  uint64_t* done;
  uint64_t seq;
  uint32_t* ctr;
  const uint64_t* tab;
  uint64_t pool;
  uint64_t units, per_wg;
  uint64_t slot_bytes, piece, kstride;
  uint32_t ppb, spans, to_paged, layers;
  uint32_t tokens, heads, row_bytes, elem;  // head-major blocks: a piece is one unit (spans = 1)
  uint64_t layer_ptr[kMaxLayers];
};

// Arguments of a self-contained launch (every entry of a linear transfer, no
// copy engine): entry w = {source, destination, bytes} goes to wave w, whose
// done tag is done[w]. N is the capacity, n the entries used.
template <uint32_t N>
struct WholeArgs {
  uint64_t* done;
  uint64_t seq;
  uint32_t n;
  uint32_t release_each;    // 1: system-scope release before each done tag
  uint64_t e[N][3];
};

// KV fetch that allocates nothing (mma_kv_fetch_noalloc): its block table and
// claim counter live in one array of the library's device code, `scratch`, of
// kNoallocScratchBytes per GPU: word 0 is the claim counter, the table (host
// slot | GPU block << 32 per block) starts at byte kNoallocTabOffset. The table
// reaches it through launches of mma_kv_noalloc_table_kernel whose arguments
// carry kNoallocTabChunk entries each; then one launch of
// mma_kv_noalloc_kernel moves the pieces, its waves claiming per_claim pieces
// at a time from the counter.
constexpr uint32_t kNoallocMaxBlocks = 65536;
constexpr uint32_t kNoallocTabOffset = 256;
constexpr uint64_t kNoallocScratchBytes = kNoallocTabOffset + 8ull * kNoallocMaxBlocks;
constexpr uint32_t kNoallocTabChunk = 448;

struct NoallocTabArgs {
  uint64_t* scratch;  // device address of the scratch array
  uint32_t first;     // table entries [first, first + count)
  uint32_t count;
  uint32_t reset;     // 1: also return the claim counter to 0 (the first launch of a call)
  uint32_t pad;
  uint64_t e[kNoallocTabChunk];
};

struct NoallocArgs {
  uint64_t* scratch;
  uint64_t pool;        // device address of the pool
  uint64_t slot_bytes, piece, kstride;
  uint64_t units;       // pieces to move: blocks * ppb
  uint32_t ppb;         // pieces per block (2 per layer: K, V)
  uint32_t per_claim;   // pieces per claim
  uint32_t layout, tokens, heads, row_bytes, elem, lds_wave;  // GPU block layout and its geometry
  uint64_t layer_ptr[kMaxLayers];
};

// constexpr: usable from host and device code alike.
constexpr uint64_t make_tag(uint64_t seq, uint64_t ticket) { return (seq << 32) | (ticket + 1); }

}  // namespace mma

#endif  // MMA_PROTO_H_
