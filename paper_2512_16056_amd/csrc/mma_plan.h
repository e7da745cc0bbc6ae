// Micro-transfer planner (Section 3.4, Task Manager) and argument checks.
// Pure host C++: no HIP, no HSA, so it can be unit-tested on any CPU.
#ifndef MMA_PLAN_H_
#define MMA_PLAN_H_

#include <stdint.h>

#include <utility>
#include <vector>

namespace mma {

struct PlanItem {
  uint64_t item;    // tensor index (list) or table index (KV)
  uint64_t offset;  // byte offset in the tensor (list) or first piece (KV)
  uint64_t bytes;   // bytes (list) or piece count (KV)
  uint32_t flags;   // kPlanCuOnly
};

constexpr uint32_t kPlanCuOnly = 1u;
constexpr uint32_t kPlanSdmaOnly = 2u;  // static-split baseline: reserved for the SDMA engines

// Static-split baseline: task i of n goes to the CU path iff the running share
// floor((i + 1) * pct / 100) grows at i, so exactly floor(n * pct / 100) tasks,
// evenly interleaved, are CU tasks.
inline bool static_cu_task(uint64_t i, uint32_t pct) { return (i + 1) * pct / 100 > i * pct / 100; }

// Fixed chunks from offset 0 of each tensor, the last one shorter; a tensor below
// `fallback` bytes is a single micro-task, below `small` it is CU-path-only.
void plan_list(const uint64_t* sizes, uint64_t n, uint64_t chunk, uint64_t fallback, uint64_t small,
               std::vector<PlanItem>& out);

// Per table entry, consecutive pieces in groups of max(1, chunk / piece_bytes).
void plan_kv(uint64_t n_blocks, uint32_t pieces_per_block, uint64_t piece_bytes, uint64_t chunk,
             std::vector<PlanItem>& out);

// Entries in range and destinations distinct.
bool tables_valid(const int32_t* src, uint32_t src_count, const int32_t* dst, uint32_t dst_count, uint64_t n);

// Half-open [begin, end) ranges pairwise disjoint (empty ranges ignored).
bool ranges_disjoint(std::vector<std::pair<uint64_t, uint64_t>> ranges);

// Byte sizes that a paged-KV layout implies (one piece, one host slot, the host
// pool, one GPU layer tensor). False if a field is 0, there are more than
// max_layers layers, a piece exceeds 4 GiB, or a size does not fit 64 bits:
// every size is a product of caller-given fields, and a wrapped product would
// let range checks pass for a smaller footprint than the kernels address.
struct KvSizes {
  uint64_t piece, slot, pool, layer;
};
bool kv_sizes(uint32_t num_layers, uint32_t block_tokens, uint32_t kv_heads, uint32_t head_dim, uint32_t elem_bytes,
              uint32_t gpu_num_blocks, uint32_t host_num_slots, uint32_t max_layers, KvSizes* out);

}  // namespace mma

#endif  // MMA_PLAN_H_
