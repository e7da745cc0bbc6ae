// Raw link probes for the measured PCIe peak, per direction. Each probe moves
// one contiguous buffer between pinned host memory and HBM without the
// multipath planner, records, engine thread or dummy kernel:
//   native_zero_copy  - a bare grid-stride streaming kernel (CU loads from
//                       pinned host memory, or stores to it), grid chosen by
//                       the caller's sweep;
//   native_sdma_all   - the buffer split evenly over a set of SDMA engines,
//                       one ROCr command each, all in flight at once;
//   native_hbm_copy   - for the measured HBM peak: a device-to-device streaming
//                       copy in wave-contiguous spans.
// Together with one plain hipMemcpyAsync they bound what the link delivers on
// this machine (the paper quotes 52-60 GB/s typical for a 64 GB/s PCIe 5.0 x16
// link, Section 2.2). Built into libmma_native.so, not into libmma.so.
#include <hip/hip_runtime.h>
#include <hsa/hsa.h>
#include <hsa/hsa_ext_amd.h>
#include <stdint.h>

#include <chrono>

namespace {

typedef unsigned int v4u __attribute__((ext_vector_type(4)));

// 8 independent 16-byte loads per thread before the matching stores.
__global__ __launch_bounds__(256) void zero_copy_stream_kernel(const v4u* __restrict__ src, v4u* __restrict__ dst,
                                                               uint64_t n16) {
  const uint64_t stride = static_cast<uint64_t>(gridDim.x) * blockDim.x;
  uint64_t i = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  for (; i + 7 * stride < n16; i += 8 * stride) {
    v4u r0 = src[i], r1 = src[i + stride], r2 = src[i + 2 * stride], r3 = src[i + 3 * stride];
    v4u r4 = src[i + 4 * stride], r5 = src[i + 5 * stride], r6 = src[i + 6 * stride], r7 = src[i + 7 * stride];
    dst[i] = r0;
    dst[i + stride] = r1;
    dst[i + 2 * stride] = r2;
    dst[i + 3 * stride] = r3;
    dst[i + 4 * stride] = r4;
    dst[i + 5 * stride] = r5;
    dst[i + 6 * stride] = r6;
    dst[i + 7 * stride] = r7;
  }
  for (; i < n16; i += stride) dst[i] = src[i];
}

// HBM-to-HBM streaming copy for the measured HBM peak: each wave moves whole
// 16 KiB spans (16 independent 16-byte loads per lane, nontemporal, before the
// matching stores), spans strided over the grid; units past the last whole span
// go one per lane.
__global__ __launch_bounds__(256) void hbm_span_copy_kernel(const v4u* __restrict__ src, v4u* __restrict__ dst,
                                                            uint64_t n16) {
  constexpr uint32_t kV = 16;
  const uint32_t lane = threadIdx.x & 63u;
  const uint64_t wave = static_cast<uint64_t>(blockIdx.x) * 4 + threadIdx.x / 64;
  const uint64_t waves = static_cast<uint64_t>(gridDim.x) * 4;
  const uint64_t span = kV * 64ull;
  const uint64_t full = n16 / span;
  for (uint64_t c = wave; c < full; c += waves) {
    const uint64_t b = c * span + lane;
    v4u v[kV];
#pragma unroll
    for (uint32_t i = 0; i < kV; ++i) v[i] = __builtin_nontemporal_load(src + b + i * 64);
#pragma unroll
    for (uint32_t i = 0; i < kV; ++i) __builtin_nontemporal_store(v[i], dst + b + i * 64);
  }
  for (uint64_t i = full * span + wave * 64 + lane; i < n16; i += waves * 64) dst[i] = src[i];
}

struct ProbeAgents {
  uint32_t bdf = 0, domain = 0;
  hsa_agent_t gpu{}, cpu{};
  bool have_gpu = false, have_cpu = false;
};

hsa_status_t probe_agent_cb(hsa_agent_t a, void* d) {
  ProbeAgents* p = static_cast<ProbeAgents*>(d);
  hsa_device_type_t t;
  if (hsa_agent_get_info(a, HSA_AGENT_INFO_DEVICE, &t) != HSA_STATUS_SUCCESS) return HSA_STATUS_SUCCESS;
  if (t == HSA_DEVICE_TYPE_CPU && !p->have_cpu) {
    p->cpu = a;
    p->have_cpu = true;
  } else if (t == HSA_DEVICE_TYPE_GPU && !p->have_gpu) {
    uint32_t bdf = 0, dom = 0;
    hsa_agent_get_info(a, static_cast<hsa_agent_info_t>(HSA_AMD_AGENT_INFO_BDFID), &bdf);
    hsa_agent_get_info(a, static_cast<hsa_agent_info_t>(HSA_AMD_AGENT_INFO_DOMAIN), &dom);
    if (bdf == p->bdf && dom == p->domain) {
      p->gpu = a;
      p->have_gpu = true;
    }
  }
  return HSA_STATUS_SUCCESS;
}

}  // namespace

extern "C" {

// dir 0: host -> device (src pinned host, dst device); 1: device -> host. Both
// pointers may also be device memory (an HBM-to-HBM streaming copy).
// bytes must be a multiple of 16 and both pointers 16-byte aligned; grid > 0.
// Returns 0 or the hipError_t of the launch.
int native_zero_copy(void* dst, const void* src, uint64_t bytes, int dir, uint32_t grid, void* stream) {
  (void)dir;  // the kernel is the same: pinned host memory is addressed directly
  if ((bytes & 15u) || (reinterpret_cast<uintptr_t>(dst) & 15u) || (reinterpret_cast<uintptr_t>(src) & 15u) ||
      grid == 0)
    return static_cast<int>(hipErrorInvalidValue);
  zero_copy_stream_kernel<<<grid, 256, 0, static_cast<hipStream_t>(stream)>>>(static_cast<const v4u*>(src),
                                                                              static_cast<v4u*>(dst), bytes >> 4);
  return static_cast<int>(hipGetLastError());
}

// HBM-to-HBM copy with hbm_span_copy_kernel on `grid` workgroups of 256
// threads; the same argument rules and return value as native_zero_copy.
int native_hbm_copy(void* dst, const void* src, uint64_t bytes, uint32_t grid, void* stream) {
  if ((bytes & 15u) || (reinterpret_cast<uintptr_t>(dst) & 15u) || (reinterpret_cast<uintptr_t>(src) & 15u) ||
      grid == 0)
    return static_cast<int>(hipErrorInvalidValue);
  hbm_span_copy_kernel<<<grid, 256, 0, static_cast<hipStream_t>(stream)>>>(static_cast<const v4u*>(src),
                                                                           static_cast<v4u*>(dst), bytes >> 4);
  return static_cast<int>(hipGetLastError());
}

// Splits [0, bytes) into popcount(engine_mask) equal 4 KiB-aligned parts (the
// last one takes the rest) and issues part e on SDMA engine e, all at once,
// then waits for every part. *out_ns = host time from the first submission to
// the last completion. The caller synchronises its streams first. Returns 0,
// -1 (no ROCr agent / bad argument) or the failing hsa_status_t.
int native_sdma_all(void* dst, const void* src, uint64_t bytes, int dir, uint32_t engine_mask, int hip_device,
                    uint64_t* out_ns) {
  if (!engine_mask || (engine_mask >> 16) || !out_ns || (dir != 0 && dir != 1)) return -1;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, hip_device) != hipSuccess) return -1;
  if (hsa_init() != HSA_STATUS_SUCCESS) return -1;
  ProbeAgents ag;
  ag.bdf = static_cast<uint32_t>((prop.pciBusID << 8) | (prop.pciDeviceID << 3));
  ag.domain = static_cast<uint32_t>(prop.pciDomainID);
  hsa_iterate_agents(probe_agent_cb, &ag);
  if (!ag.have_gpu || !ag.have_cpu) {
    hsa_shut_down();
    return -1;
  }
  const hsa_agent_t dst_agent = dir == 0 ? ag.gpu : ag.cpu;
  const hsa_agent_t src_agent = dir == 0 ? ag.cpu : ag.gpu;
  const uint32_t parts = static_cast<uint32_t>(__builtin_popcount(engine_mask));
  const uint64_t per = (bytes / parts) & ~4095ull;
  if (per == 0) {
    hsa_shut_down();
    return -1;
  }
  hsa_signal_t sig[16];
  uint32_t made = 0;
  int rc = 0;
  for (; made < parts; ++made) {
    if (hsa_signal_create(1, 0, nullptr, &sig[made]) != HSA_STATUS_SUCCESS) {
      rc = -1;
      break;
    }
  }
  const auto t0 = std::chrono::steady_clock::now();
  uint32_t issued = 0;
  for (uint32_t e = 0, k = 0; rc == 0 && e < 16; ++e) {
    if (!(engine_mask & (1u << e))) continue;
    const uint64_t off = k * per;
    const uint64_t n = k + 1 == parts ? bytes - off : per;
    const hsa_status_t s = hsa_amd_memory_async_copy_on_engine(
        static_cast<uint8_t*>(dst) + off, dst_agent, static_cast<const uint8_t*>(src) + off, src_agent, n, 0,
        nullptr, sig[k], static_cast<hsa_amd_sdma_engine_id_t>(1u << e), false);
    if (s != HSA_STATUS_SUCCESS) rc = static_cast<int>(s);
    else ++issued;
    ++k;
  }
  for (uint32_t k = 0; k < issued; ++k)
    hsa_signal_wait_scacquire(sig[k], HSA_SIGNAL_CONDITION_LT, 1, UINT64_MAX, HSA_WAIT_STATE_ACTIVE);
  const auto t1 = std::chrono::steady_clock::now();
  *out_ns = static_cast<uint64_t>(std::chrono::duration_cast<std::chrono::nanoseconds>(t1 - t0).count());
  for (uint32_t k = 0; k < made; ++k) hsa_signal_destroy(sig[k]);
  hsa_shut_down();
  return rc;
}

}  // extern "C"
