// Micro-transfer planner and argument checks (host-only).
#include "mma_plan.h"

#include <algorithm>
#include <new>

#include "../../include/mma.h"

namespace mma {

// Room for `count` more items, or std::bad_alloc at once: a count beyond what
// memory can hold fails here instead of after growing the vector for a while.
static void reserve_more(std::vector<PlanItem>& out, uint64_t count) {
  if (count > out.max_size() - out.size()) throw std::bad_alloc();
  out.reserve(out.size() + count);
}

void plan_list(const uint64_t* sizes, uint64_t n, uint64_t chunk, uint64_t fallback, uint64_t small,
               std::vector<PlanItem>& out) {
  uint64_t count = 0;  // saturates: only compared with what a vector can hold
  for (uint64_t t = 0; t < n; ++t) {
    const uint64_t sz = sizes[t], c = sz == 0 ? 0 : sz < fallback ? 1 : sz / chunk + (sz % chunk != 0);
    count = c > UINT64_MAX - count ? UINT64_MAX : count + c;
  }
  reserve_more(out, count);
  for (uint64_t t = 0; t < n; ++t) {
    const uint64_t sz = sizes[t];
    if (sz == 0) continue;
    const uint32_t flags = sz < small ? kPlanCuOnly : 0u;
    if (sz < fallback) {
      out.push_back({t, 0, sz, flags});
      continue;
    }
    for (uint64_t o = 0; o < sz;) {  // advances by what is left at the end: o never wraps
      const uint64_t b = std::min(chunk, sz - o);
      out.push_back({t, o, b, flags});
      o += b;
    }
  }
}

void plan_kv(uint64_t n_blocks, uint32_t pieces_per_block, uint64_t piece_bytes, uint64_t chunk,
             std::vector<PlanItem>& out) {
  uint64_t per = piece_bytes ? chunk / piece_bytes : 1;
  if (per < 1) per = 1;
  const uint64_t groups = pieces_per_block / per + (pieces_per_block % per != 0);
  reserve_more(out, groups && n_blocks > UINT64_MAX / groups ? UINT64_MAX : n_blocks * groups);
  for (uint64_t i = 0; i < n_blocks; ++i)
    for (uint64_t p = 0; p < pieces_per_block; p += per)
      out.push_back({i, p, std::min<uint64_t>(per, pieces_per_block - p), 0u});
}

bool tables_valid(const int32_t* src, uint32_t src_count, const int32_t* dst, uint32_t dst_count, uint64_t n) {
  for (uint64_t i = 0; i < n; ++i) {
    if (src[i] < 0 || static_cast<uint32_t>(src[i]) >= src_count) return false;
    if (dst[i] < 0 || static_cast<uint32_t>(dst[i]) >= dst_count) return false;
  }
  if (n < 2) return true;
  // Distinct destinations. A short table against a large cache (a few blocks
  // fetched into millions) sorts a copy of its n entries rather than clearing
  // a flag per destination block on every call.
  if (n < dst_count / 64) {
    std::vector<int32_t> d(dst, dst + n);
    std::sort(d.begin(), d.end());
    return std::adjacent_find(d.begin(), d.end()) == d.end();
  }
  std::vector<uint8_t> seen(dst_count, 0);
  for (uint64_t i = 0; i < n; ++i) {
    if (seen[dst[i]]) return false;
    seen[dst[i]] = 1;
  }
  return true;
}

bool ranges_disjoint(std::vector<std::pair<uint64_t, uint64_t>> r) {
  r.erase(std::remove_if(r.begin(), r.end(), [](const auto& x) { return x.second <= x.first; }), r.end());
  std::sort(r.begin(), r.end());
  for (size_t i = 1; i < r.size(); ++i)
    if (r[i].first < r[i - 1].second) return false;
  return true;
}

bool kv_sizes(uint32_t num_layers, uint32_t block_tokens, uint32_t kv_heads, uint32_t head_dim, uint32_t elem_bytes,
              uint32_t gpu_num_blocks, uint32_t host_num_slots, uint32_t max_layers, KvSizes* out) {
  if (!num_layers || num_layers > max_layers || !block_tokens || !kv_heads || !head_dim || !elem_bytes ||
      !gpu_num_blocks || !host_num_slots)
    return false;
  uint64_t piece = block_tokens, slot = 0, pool = 0, layer = 0;
  if (__builtin_mul_overflow(piece, static_cast<uint64_t>(kv_heads), &piece) ||
      __builtin_mul_overflow(piece, static_cast<uint64_t>(head_dim), &piece) ||
      __builtin_mul_overflow(piece, static_cast<uint64_t>(elem_bytes), &piece) || piece > (1ull << 32))
    return false;
  slot = piece * 2 * num_layers;  // at most 2^32 * 2 * max_layers
  if (__builtin_mul_overflow(slot, static_cast<uint64_t>(host_num_slots), &pool) ||
      __builtin_mul_overflow(2 * piece, static_cast<uint64_t>(gpu_num_blocks), &layer))
    return false;
  *out = {piece, slot, pool, layer};
  return true;
}

}  // namespace mma

// A C++ exception never leaves these calls (a C caller cannot catch it): the
// planners and the table check allocate, and running out of host memory is
// MMA_ERR_NO_MEMORY.
extern "C" {

mma_status_t mma_plan_list(const uint64_t* sizes, uint64_t n, uint64_t chunk, uint64_t fallback, uint64_t small,
                           mma_plan_entry_t* out, uint64_t cap, uint64_t* n_out) try {
  if (!n_out || chunk == 0 || (n && !sizes)) return MMA_ERR_INVALID_ARG;
  std::vector<mma::PlanItem> v;
  mma::plan_list(sizes, n, chunk, fallback, small, v);
  *n_out = v.size();
  if (!out) return cap == 0 ? MMA_OK : MMA_ERR_INVALID_ARG;
  if (cap < v.size()) return MMA_ERR_BUFFER_TOO_SMALL;
  for (size_t i = 0; i < v.size(); ++i) out[i] = {v[i].item, v[i].offset, v[i].bytes, v[i].flags, 0u};
  return MMA_OK;
} catch (const std::bad_alloc&) {
  return MMA_ERR_NO_MEMORY;
} catch (...) {
  return MMA_ERR_INTERNAL;
}

mma_status_t mma_plan_kv(uint64_t n_blocks, uint32_t pieces_per_block, uint64_t piece_bytes, uint64_t chunk,
                         mma_plan_entry_t* out, uint64_t cap, uint64_t* n_out) try {
  if (!n_out || chunk == 0 || piece_bytes == 0) return MMA_ERR_INVALID_ARG;
  std::vector<mma::PlanItem> v;
  mma::plan_kv(n_blocks, pieces_per_block, piece_bytes, chunk, v);
  *n_out = v.size();
  if (!out) return cap == 0 ? MMA_OK : MMA_ERR_INVALID_ARG;
  if (cap < v.size()) return MMA_ERR_BUFFER_TOO_SMALL;
  for (size_t i = 0; i < v.size(); ++i) out[i] = {v[i].item, v[i].offset, v[i].bytes, v[i].flags, 0u};
  return MMA_OK;
} catch (const std::bad_alloc&) {
  return MMA_ERR_NO_MEMORY;
} catch (...) {
  return MMA_ERR_INTERNAL;
}

mma_status_t mma_kv_layout_sizes(const mma_kv_layout_t* layout, uint64_t* piece_bytes, uint64_t* slot_bytes,
                                 uint64_t* pool_bytes, uint64_t* layer_bytes) {
  mma::KvSizes z;
  if (!layout || !mma::kv_sizes(layout->num_layers, layout->block_tokens, layout->kv_heads, layout->head_dim,
                                layout->elem_bytes, layout->gpu_num_blocks, layout->host_num_slots,
                                MMA_MAX_LAYERS, &z))
    return MMA_ERR_INVALID_ARG;
  if (piece_bytes) *piece_bytes = z.piece;
  if (slot_bytes) *slot_bytes = z.slot;
  if (pool_bytes) *pool_bytes = z.pool;
  if (layer_bytes) *layer_bytes = z.layer;
  return MMA_OK;
}

mma_status_t mma_validate_kv_tables(const int32_t* src, uint32_t src_count, const int32_t* dst, uint32_t dst_count,
                                    uint64_t n) try {
  if (n && (!src || !dst)) return MMA_ERR_INVALID_ARG;
  return mma::tables_valid(src, src_count, dst, dst_count, n) ? MMA_OK : MMA_ERR_INVALID_ARG;
} catch (const std::bad_alloc&) {
  return MMA_ERR_NO_MEMORY;
} catch (...) {
  return MMA_ERR_INTERNAL;
}

}  // extern "C"
