// Native single-path comparators for the benchmark: the same transfers issued as
// plain hipMemcpyAsync calls on one stream (the paper's baseline, Section 5:
// native copies statically bound to the GPU's own PCIe path). Not part of the
// multipath path; built as its own library (libmma_native.so).
#include <dlfcn.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

extern "C" {

// Per-piece hipMemcpyAsync KV fetch: n blocks x L layers x {K, V}.
int native_kv_fetch(const void* host_pool, void* const* layers, const int32_t* host_slots, const int32_t* gpu_blocks,
                    uint64_t n, uint32_t num_layers, uint64_t piece, uint64_t gpu_num_blocks, void* stream) {
  const uint64_t slot = 2ull * num_layers * piece;
  for (uint64_t i = 0; i < n; ++i)
    for (uint32_t l = 0; l < num_layers; ++l)
      for (uint32_t k = 0; k < 2; ++k) {
        const uint8_t* src = static_cast<const uint8_t*>(host_pool) + host_slots[i] * slot + (2 * l + k) * piece;
        uint8_t* dst = static_cast<uint8_t*>(layers[l]) + (k * gpu_num_blocks + gpu_blocks[i]) * piece;
        hipError_t e = hipMemcpyAsync(dst, src, piece, hipMemcpyHostToDevice, static_cast<hipStream_t>(stream));
        if (e != hipSuccess) return static_cast<int>(e);
      }
  return 0;
}

int native_kv_offload(void* host_pool, void* const* layers, const int32_t* gpu_blocks, const int32_t* host_slots,
                      uint64_t n, uint32_t num_layers, uint64_t piece, uint64_t gpu_num_blocks, void* stream) {
  const uint64_t slot = 2ull * num_layers * piece;
  for (uint64_t j = 0; j < n; ++j)
    for (uint32_t l = 0; l < num_layers; ++l)
      for (uint32_t k = 0; k < 2; ++k) {
        uint8_t* dst = static_cast<uint8_t*>(host_pool) + host_slots[j] * slot + (2 * l + k) * piece;
        const uint8_t* src = static_cast<const uint8_t*>(layers[l]) + (k * gpu_num_blocks + gpu_blocks[j]) * piece;
        hipError_t e = hipMemcpyAsync(dst, src, piece, hipMemcpyDeviceToHost, static_cast<hipStream_t>(stream));
        if (e != hipSuccess) return static_cast<int>(e);
      }
  return 0;
}

// The same per-piece fetch as one batched call, when the HIP runtime in the
// process provides hipMemcpyBatchAsync; returns -1 if it does not.
int native_kv_fetch_batch(const void* host_pool, void* const* layers, const int32_t* host_slots,
                          const int32_t* gpu_blocks, uint64_t n, uint32_t num_layers, uint64_t piece,
                          uint64_t gpu_num_blocks, void* stream) {
  typedef hipError_t (*batch_fn)(void**, void**, size_t*, size_t, void*, size_t*, size_t, size_t*, hipStream_t);
  static batch_fn fn = reinterpret_cast<batch_fn>(dlsym(RTLD_DEFAULT, "hipMemcpyBatchAsync"));
  if (!fn) return -1;
  const uint64_t slot = 2ull * num_layers * piece;
  std::vector<void*> d, s;
  std::vector<size_t> z;
  for (uint64_t i = 0; i < n; ++i)
    for (uint32_t l = 0; l < num_layers; ++l)
      for (uint32_t k = 0; k < 2; ++k) {
        s.push_back(const_cast<uint8_t*>(static_cast<const uint8_t*>(host_pool)) + host_slots[i] * slot +
                    (2 * l + k) * piece);
        d.push_back(static_cast<uint8_t*>(layers[l]) + (k * gpu_num_blocks + gpu_blocks[i]) * piece);
        z.push_back(piece);
      }
  size_t fail_idx = 0;
  hipError_t e = fn(d.data(), s.data(), z.data(), d.size(), nullptr, nullptr, 0, &fail_idx,
                    static_cast<hipStream_t>(stream));
  return static_cast<int>(e);
}

// A list of independent copies, one hipMemcpyAsync each.
int native_list(void* const* dsts, const void* const* srcs, const uint64_t* sizes, uint64_t n, int dir, void* stream) {
  const hipMemcpyKind kind = dir == 0 ? hipMemcpyHostToDevice : hipMemcpyDeviceToHost;
  for (uint64_t i = 0; i < n; ++i) {
    hipError_t e = hipMemcpyAsync(dsts[i], srcs[i], sizes[i], kind, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return static_cast<int>(e);
  }
  return 0;
}

}  // extern "C"
