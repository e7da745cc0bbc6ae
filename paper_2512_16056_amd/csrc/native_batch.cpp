// Native batched comparator for the 64k-token KV fetch: every (block, layer,
// K/V) piece of the fetch as one entry of a single hipMemcpyBatchAsync call
// (the runtime's own batched host-to-device copy), timed with HIP events on
// one stream. It is a program of its own because the HIP runtime that torch
// loads does not export hipMemcpyBatchAsync; this one links the system ROCm
// runtime, runs before the benchmark process touches the GPU, and prints one
// JSON line. Not part of the multipath path.
//
// Usage: native_batch TABLES N_BLOCKS LAYERS PIECE_BYTES GPU_NUM_BLOCKS HOST_NUM_SLOTS REPS
//   TABLES: raw int32 host_slots[N_BLOCKS] followed by gpu_blocks[N_BLOCKS].
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <string>
#include <vector>

namespace {

int report_error(const char* what, hipError_t e, size_t fail_idx) {
  printf("{\"available\": true, \"ok\": false, \"call\": \"%s\", \"error\": \"%s\", \"code\": %d, \"fail_idx\": %zu}\n",
         what, hipGetErrorString(e), static_cast<int>(e), fail_idx);
  return 0;  // the comparator ran; the runtime's answer is the result
}

}  // namespace

int main(int argc, char** argv) {
  if (argc != 8) {
    fprintf(stderr, "usage: %s TABLES N_BLOCKS LAYERS PIECE_BYTES GPU_NUM_BLOCKS HOST_NUM_SLOTS REPS\n", argv[0]);
    return 2;
  }
  const uint64_t n = strtoull(argv[2], nullptr, 0), layers = strtoull(argv[3], nullptr, 0);
  const uint64_t piece = strtoull(argv[4], nullptr, 0), nb = strtoull(argv[5], nullptr, 0);
  const uint64_t slots = strtoull(argv[6], nullptr, 0);
  const int reps = atoi(argv[7]);
  std::vector<int32_t> tab(2 * n);
  FILE* f = fopen(argv[1], "rb");
  if (!f || fread(tab.data(), sizeof(int32_t), 2 * n, f) != 2 * n) {
    fprintf(stderr, "cannot read %s\n", argv[1]);
    return 2;
  }
  fclose(f);
  const int32_t* hs = tab.data();
  const int32_t* gb = tab.data() + n;
  for (uint64_t i = 0; i < n; ++i)
    if (hs[i] < 0 || static_cast<uint64_t>(hs[i]) >= slots || gb[i] < 0 || static_cast<uint64_t>(gb[i]) >= nb) {
      fprintf(stderr, "table entry %llu out of range\n", static_cast<unsigned long long>(i));
      return 2;
    }
  const uint64_t slot_bytes = 2 * layers * piece, layer_bytes = 2 * nb * piece;
  hipError_t e = hipSetDevice(0);
  if (e != hipSuccess) return report_error("hipSetDevice", e, 0);
  uint8_t* pool = nullptr;
  if ((e = hipHostMalloc(reinterpret_cast<void**>(&pool), slots * slot_bytes, hipHostMallocDefault)) != hipSuccess)
    return report_error("hipHostMalloc", e, 0);
  // every slot's bytes name the slot, so a sampled piece shows where it came from
  for (uint64_t s = 0; s < slots; ++s) memset(pool + s * slot_bytes, static_cast<int>(s * 37 + 11) & 0xFF, slot_bytes);
  std::vector<uint8_t*> dev(layers, nullptr);
  for (uint64_t l = 0; l < layers; ++l)
    if ((e = hipMalloc(reinterpret_cast<void**>(&dev[l]), layer_bytes)) != hipSuccess)
      return report_error("hipMalloc", e, 0);
  const uint64_t count = n * layers * 2;
  std::vector<void*> dsts(count), srcs(count);
  std::vector<size_t> sizes(count, piece);
  uint64_t c = 0;
  for (uint64_t i = 0; i < n; ++i)
    for (uint64_t l = 0; l < layers; ++l)
      for (uint64_t k = 0; k < 2; ++k, ++c) {
        srcs[c] = pool + hs[i] * slot_bytes + (2 * l + k) * piece;
        dsts[c] = dev[l] + (k * nb + gb[i]) * piece;
      }
  hipStream_t st;
  if ((e = hipStreamCreateWithFlags(&st, hipStreamNonBlocking)) != hipSuccess)
    return report_error("hipStreamCreate", e, 0);
  // Attribute sets tried in turn until the runtime accepts one: none (the header marks attributes
  // unsupported), then stream-ordered source access with location hints (host source, device
  // destination), then unordered source access with the same hints.
  hipMemcpyAttributes attrs[3];
  memset(attrs, 0, sizeof attrs);
  attrs[1].srcAccessOrder = hipMemcpySrcAccessOrderStream;
  attrs[1].srcLocHint.type = hipMemLocationTypeHost;
  attrs[1].dstLocHint.type = hipMemLocationTypeDevice;
  attrs[1].dstLocHint.id = 0;
  attrs[2] = attrs[1];
  attrs[2].srcAccessOrder = hipMemcpySrcAccessOrderAny;
  const char* names[3] = {"no attributes", "stream-ordered source, host->device hints",
                          "any-order source, host->device hints"};
  int chosen = -1;
  std::string tried;
  for (int k = 0; k < 3 && chosen < 0; ++k) {
    size_t fail_idx = 0, idx = 0;
    // valid attribute and index pointers even when none is passed (numAttrs 0)
    e = hipMemcpyBatchAsync(dsts.data(), srcs.data(), sizes.data(), count, &attrs[k], &idx, k ? 1 : 0, &fail_idx, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e == hipSuccess) {
      chosen = k;
    } else {
      (void)hipGetLastError();
      tried += std::string(tried.empty() ? "" : "; ") + names[k] + ": " + hipGetErrorString(e);
    }
  }
  if (chosen < 0) {
    printf("{\"available\": true, \"ok\": false, \"call\": \"hipMemcpyBatchAsync\", \"error\": \"%s\"}\n",
           tried.c_str());
    return 0;
  }
  size_t attr_idx = 0;
  hipEvent_t a, b;
  hipEventCreate(&a);
  hipEventCreate(&b);
  std::vector<float> ms;
  for (int r = 0; r < reps; ++r) {  // the accepted call above warmed up
    size_t fail_idx = 0;
    hipEventRecord(a, st);
    e = hipMemcpyBatchAsync(dsts.data(), srcs.data(), sizes.data(), count, &attrs[chosen], &attr_idx, chosen ? 1 : 0,
                            &fail_idx, st);
    if (e != hipSuccess) return report_error("hipMemcpyBatchAsync", e, fail_idx);
    hipEventRecord(b, st);
    if ((e = hipEventSynchronize(b)) != hipSuccess) return report_error("hipEventSynchronize", e, 0);
    float t = 0;
    hipEventElapsedTime(&t, a, b);
    ms.push_back(t);
  }
  // sampled check: 64 pieces spread over the batch hold their source slot's byte
  bool ok = true;
  std::vector<uint8_t> back(piece);
  for (uint64_t s = 0; s < 64; ++s) {
    const uint64_t j = (s * 4099) % count;
    if (hipMemcpy(back.data(), dsts[j], piece, hipMemcpyDeviceToHost) != hipSuccess) {
      ok = false;
      break;
    }
    const uint64_t i = j / (2 * layers);
    const uint8_t want = static_cast<uint8_t>(static_cast<uint64_t>(hs[i]) * 37 + 11);
    ok = ok && std::all_of(back.begin(), back.end(), [&](uint8_t v) { return v == want; });
  }
  std::sort(ms.begin(), ms.end());
  printf("{\"available\": true, \"ok\": %s, \"entries\": %llu, \"bytes\": %llu, \"ms_median\": %.3f, "
         "\"ms_min\": %.3f, \"ms_max\": %.3f, \"reps\": %d, \"attributes\": \"%s\", \"refused\": \"%s\", "
         "\"runtime\": %d}\n",
         ok ? "true" : "false", static_cast<unsigned long long>(count),
         static_cast<unsigned long long>(count * piece), ms[ms.size() / 2], ms.front(), ms.back(), reps,
         names[chosen], tried.c_str(), HIP_VERSION);
  for (uint64_t l = 0; l < layers; ++l) hipFree(dev[l]);
  hipHostFree(pool);
  return 0;
}
