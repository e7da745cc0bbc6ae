// Device side of the multipath copy path for gfx950 (MI355X).
//
// mma_transfer_kernel is the per-transfer "dummy task" (Section 3.3, Sync
// Engine; Section 4, Spin Kernel) enqueued on the caller's stream in place of
// the copy. Its waves do three things:
//   1. the first wave to run publishes `started` -- the stream -> engine start
//      signal (the paper uses a host callback for this direction);
//   2. every wave is a worker of the CU path (Section 3.4: one outstanding
//      queue per path): it claims ring entries with a device-memory atomic and
//      moves them with wide zero-copy loads/stores across PCIe, or between the
//      paged KV layout and SDMA staging buffers in HBM; each wave signals its
//      own completions (wavefront-level completion);
//   3. the last wave to finish claiming holds the stream until the engine
//      reports that every micro-task of every path has landed (the spin wait
//      of Section 4), with a bounded, progress-re-armed watchdog, then exits
//      and releases downstream stream work.
//
// mma_digest_kernel is the dependent HBM-bound check kernel of the
// mixed-contention workload.
#include <hip/hip_runtime.h>

#include "mma_proto.h"

namespace mma {
namespace {

constexpr int kUnroll = 16;  // 16 x 16 B loads in flight per lane (wave_copy spells them out)

// Global-address-space views: global_load/global_store instead of flat ones
// (no LDS counter waits on the copy path).
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) u32x4 gu4;

__device__ __forceinline__ uint64_t ld_sys(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}
__device__ __forceinline__ uint32_t ld_sys32(const uint32_t* p) {
  return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}
__device__ __forceinline__ void st_sys(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Wave-cooperative copy of n bytes. Consecutive lanes move consecutive 16-byte
// units, so each load instruction covers one contiguous 1 KiB span; a lane keeps
// kUnroll loads in flight before storing. Byte head/tail handle any alignment
// when src and dst are equally aligned modulo 16; otherwise a byte loop is used.
__device__ __forceinline__ void wave_copy(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
                                          uint64_t n, uint32_t lane) {
  if (((reinterpret_cast<uintptr_t>(src) ^ reinterpret_cast<uintptr_t>(dst)) & 15u) == 0) {
    uint64_t head = (16u - (reinterpret_cast<uintptr_t>(src) & 15u)) & 15u;
    if (head > n) head = n;
    if (lane < head) dst[lane] = src[lane];
    src += head;
    dst += head;
    n -= head;
    const uint64_t n16 = n >> 4;
    const gu4* s = (const gu4*)(src);  // generic -> global address space
    gu4* d = (gu4*)(dst);
    uint64_t i = lane;
    for (; i + (kUnroll - 1) * kWave < n16; i += kUnroll * kWave) {
#define MMA_LD(k) const u32x4 v##k = s[i + (k) * kWave];
#define MMA_ST(k) d[i + (k) * kWave] = v##k;
      MMA_LD(0) MMA_LD(1) MMA_LD(2) MMA_LD(3) MMA_LD(4) MMA_LD(5) MMA_LD(6) MMA_LD(7)
      MMA_LD(8) MMA_LD(9) MMA_LD(10) MMA_LD(11) MMA_LD(12) MMA_LD(13) MMA_LD(14) MMA_LD(15)
      // Keep every load of the batch in flight before the first store: the
      // scheduler would otherwise pair each load with its store and expose the
      // full PCIe latency once per 16 bytes.
      __builtin_amdgcn_sched_barrier(0);
      MMA_ST(0) MMA_ST(1) MMA_ST(2) MMA_ST(3) MMA_ST(4) MMA_ST(5) MMA_ST(6) MMA_ST(7)
      MMA_ST(8) MMA_ST(9) MMA_ST(10) MMA_ST(11) MMA_ST(12) MMA_ST(13) MMA_ST(14) MMA_ST(15)
#undef MMA_LD
#undef MMA_ST
    }
    for (; i < n16; i += kWave) d[i] = s[i];
    const uint64_t tail = n & 15u;
    const uint64_t base = n16 << 4;
    if (lane < tail) dst[base + lane] = src[base + lane];
  } else {
    for (uint64_t i = lane; i < n; i += kWave) dst[i] = src[i];
  }
}

__device__ __forceinline__ uint64_t bcast(uint64_t v) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v >> 32));
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

}  // namespace

__global__ __launch_bounds__(kBlock) void mma_transfer_kernel(KernelArgs a) {
  __shared__ uint64_t s_layer[kMaxLayers];
  Record* rec = a.rec;
  DevState* ds = a.ds;
  const uint32_t lane = threadIdx.x & (kWave - 1);

  // KV geometry: one PCIe read per workgroup, then served from LDS.
  uint32_t nl = ld_sys32(&rec->h.kv_layers);
  if (nl > kMaxLayers) nl = kMaxLayers;
  for (uint32_t i = threadIdx.x; i < nl; i += kBlock) s_layer[i] = ld_sys(&rec->h.layer_ptr[i]);
  const uint64_t piece = ld_sys(&rec->h.kv_piece_bytes);
  const uint64_t kstride = ld_sys(&rec->h.kv_kstride);
  __syncthreads();
  // Writes that precede the transfer in stream order, and host data, are visible.
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");

  // 1. start signal (stream -> engine).
  if (lane == 0) {
    const uint32_t first = __hip_atomic_fetch_add(&ds->arrived, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (first == 0) {
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "");
      st_sys(&rec->h.started, a.seq);
    }
  }

  // 2. CU-path worker loop. Lane 0 claims and polls; the wave copies.
  uint64_t hb = 0, t_prog = 0;
  uint32_t timed_out = 0;
  if (lane == 0) {
    hb = ld_sys(&rec->h.heartbeat);
    t_prog = wall_clock64();
  }
  for (;;) {
    uint64_t ea = 0, eb = 0, ck = 0, x = 0;
    uint32_t state = 0;  // 1: entry ready, 2: no more entries, 3: watchdog
    if (lane == 0) {
      x = __hip_atomic_fetch_add(&ds->cursor, static_cast<uint64_t>(1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const CuEntry* e = &rec->ring[x % kRingSize];
      const uint64_t expect = make_tag(a.seq, x);
      for (;;) {
        if (ld_sys(&e->tag) == expect) {
          state = 1;
          break;
        }
        if (ld_sys(&rec->h.closed) == a.seq && x >= ld_sys(&rec->h.cu_total)) {
          state = 2;
          break;
        }
        const uint64_t now = wall_clock64();
        const uint64_t hb2 = ld_sys(&rec->h.heartbeat);
        if (hb2 != hb) {
          hb = hb2;
          t_prog = now;
        } else if (now - t_prog > a.watchdog_ticks ||
                   __hip_atomic_load(&ds->timed_out, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) {
          state = 3;
          break;
        }
        __builtin_amdgcn_s_sleep(4);
      }
      if (state == 1) {
        ea = ld_sys(&e->a);
        eb = ld_sys(&e->b);
        ck = ld_sys(reinterpret_cast<const uint64_t*>(&e->count));
      }
    }
    state = static_cast<uint32_t>(bcast(state));
    if (state != 1) {
      if (state == 3) timed_out = 1;
      break;
    }
    x = bcast(x);
    ea = bcast(ea);
    eb = bcast(eb);
    ck = bcast(ck);
    const uint32_t count = static_cast<uint32_t>(ck);
    const uint32_t kind = static_cast<uint32_t>(ck >> 32) & kEntryKindMask;
    const uint32_t p0 = static_cast<uint32_t>(ck >> 40);
    // Data landed by an SDMA engine during this kernel: drop any stale copy of
    // it from this CU's vector L1 (and non-coherent L2 lines) before reading.
    if ((ck >> 32) & kEntryAcquire) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");

    if (kind == kEntryCopy) {
      wave_copy(reinterpret_cast<const uint8_t*>(ea), reinterpret_cast<uint8_t*>(eb), count, lane);
    } else if (kind == kEntryToPaged) {
      for (uint32_t j = 0; j < count; ++j) {
        const uint32_t p = p0 + j;
        uint8_t* dst = reinterpret_cast<uint8_t*>(s_layer[p >> 1]) + (p & 1u) * kstride + eb * piece;
        wave_copy(reinterpret_cast<const uint8_t*>(ea) + j * piece, dst, piece, lane);
      }
    } else if (kind == kEntryFromPaged) {
      for (uint32_t j = 0; j < count; ++j) {
        const uint32_t p = p0 + j;
        const uint8_t* src = reinterpret_cast<const uint8_t*>(s_layer[p >> 1]) + (p & 1u) * kstride + eb * piece;
        wave_copy(src, reinterpret_cast<uint8_t*>(ea) + j * piece, piece, lane);
      }
    }
    if (a.release_each) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "");
    if (lane == 0) {
      st_sys(&rec->done[x % kRingSize], make_tag(a.seq, x));
      t_prog = wall_clock64();
    }
  }

  // 3. leave; the last wave out waits for completion of all paths.
  if (lane == 0) {
    if (timed_out) {
      __hip_atomic_store(&ds->timed_out, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    const uint32_t n = __hip_atomic_fetch_add(&ds->exited, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    if (n == a.total_waves - 1) {
      uint32_t to = __hip_atomic_load(&ds->timed_out, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      while (!to && ld_sys(&rec->h.complete) != a.seq) {
        const uint64_t now = wall_clock64();
        const uint64_t hb2 = ld_sys(&rec->h.heartbeat);
        if (hb2 != hb) {
          hb = hb2;
          t_prog = now;
        } else if (now - t_prog > a.watchdog_ticks) {
          to = 1;
        }
        __builtin_amdgcn_s_sleep(8);
      }
      if (to) __hip_atomic_store(&rec->h.status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      __hip_atomic_store(&ds->cursor, static_cast<uint64_t>(0), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&ds->arrived, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&ds->exited, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&ds->timed_out, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "");
      st_sys(&rec->h.released, a.seq);
    }
  }
}

// digest += sum_i (w_i + 1) * (2i + 1) mod 2^64 over nw words (+ one zero-padded
// tail word of tail_len bytes at tail). vec4: w is 16-byte aligned.
__global__ __launch_bounds__(256) void mma_digest_kernel(const uint32_t* __restrict__ w, uint64_t nw,
                                                         const uint8_t* __restrict__ tail, uint32_t tail_len,
                                                         uint32_t vec4, unsigned long long* out) {
  const uint64_t tid = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const uint64_t stride = static_cast<uint64_t>(gridDim.x) * blockDim.x;
  uint64_t acc = 0;
  uint64_t done = 0;
  if (vec4) {
    const uint64_t n4 = nw >> 2;
    const uint4* w4 = reinterpret_cast<const uint4*>(w);
    for (uint64_t j = tid; j < n4; j += stride) {
      const uint4 v = w4[j];
      const uint64_t i = j << 2;
      acc += (v.x + 1ull) * (2 * i + 1) + (v.y + 1ull) * (2 * i + 3) + (v.z + 1ull) * (2 * i + 5) +
             (v.w + 1ull) * (2 * i + 7);
    }
    done = n4 << 2;
  }
  for (uint64_t i = done + tid; i < nw; i += stride) acc += (w[i] + 1ull) * (2 * i + 1);
  if (tid == 0 && tail_len) {
    uint32_t t = 0;
    for (uint32_t b = 0; b < tail_len; ++b) t |= static_cast<uint32_t>(tail[b]) << (8 * b);
    acc += (t + 1ull) * (2 * nw + 1);
  }
  for (int off = kWave / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if ((threadIdx.x & (kWave - 1)) == 0 && acc) atomicAdd(out, static_cast<unsigned long long>(acc));
}

hipError_t launch_transfer(const KernelArgs& args, uint32_t grid, hipStream_t stream) {
  KernelArgs a = args;
  void* params[] = {&a};
  return hipLaunchKernel(reinterpret_cast<const void*>(&mma_transfer_kernel), dim3(grid), dim3(kBlock), params, 0,
                         stream);
}

hipError_t launch_digest(const void* ptr, uint64_t bytes, uint64_t* out, hipStream_t stream) {
  const uint32_t* w = static_cast<const uint32_t*>(ptr);
  uint64_t nw = bytes >> 2;
  const uint8_t* tail = static_cast<const uint8_t*>(ptr) + (nw << 2);
  uint32_t tail_len = static_cast<uint32_t>(bytes & 3u);
  uint32_t vec4 = (reinterpret_cast<uintptr_t>(ptr) & 15u) == 0 ? 1u : 0u;
  unsigned long long* o = reinterpret_cast<unsigned long long*>(out);
  uint64_t want = (nw + 4095) / 4096;
  uint32_t grid = static_cast<uint32_t>(want < 1 ? 1 : (want > 2048 ? 2048 : want));
  void* params[] = {&w, &nw, &tail, &tail_len, &vec4, &o};
  return hipLaunchKernel(reinterpret_cast<const void*>(&mma_digest_kernel), dim3(grid), dim3(256), params, 0,
                         stream);
}

}  // namespace mma
