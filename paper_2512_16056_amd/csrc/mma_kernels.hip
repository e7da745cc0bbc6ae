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
// Under device control the whole CU share is in the ring before the launch
// (a ticket past it ends a wave's claims) and the last wave waits for the copy
// engines' own completion signal instead of the engine's word: no host thread
// takes part once the kernel runs. mma_transfer_xpacked_kernel<E> is the same
// kernel for the x-packed GPU block layout (an LDS transform per piece),
// mma_transfer_hnd_kernel for the head-major one (a row permutation), and
// mma_whole_kernel<N> a self-contained launch whose N entries travel in its
// arguments.
//
// Every host-memory poll is a PCIe read that competes with the payload for the
// link, so polls are few: one load instruction both checks and fetches a ring
// entry, an idle wave backs off exponentially, and the close/heartbeat words
// are read only every few polls.
//
// mma_digest_kernel is the dependent HBM-bound check kernel of the
// mixed-contention workload.
#include <hip/hip_runtime.h>

#include "mma_proto.h"
#include "mma_xpacked.h"

namespace mma {
namespace {

// Global-address-space views: global_load/global_store instead of flat ones
// (no LDS-counter waits on the copy path).
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) u32x4 gu4;

__device__ __forceinline__ uint64_t ld_sys(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}
__device__ __forceinline__ void st_sys(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

__device__ __forceinline__ uint64_t lane_u64(uint64_t v, int lane) {
  const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(v), lane);
  const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(v >> 32), lane);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ __forceinline__ void backoff(uint32_t n) {
  for (uint32_t k = 0; k < n; ++k) __builtin_amdgcn_s_sleep(8);  // ~512 cycles each
}

// One batch = 16 loads of 16 B per lane = 16 KiB per wave.
constexpr uint64_t kBatch = 16 * kWave;  // in 16-byte units

#define MMA_LOAD16(V, base)                                                                                \
  V##0 = s[(base) + 0 * kWave]; V##1 = s[(base) + 1 * kWave]; V##2 = s[(base) + 2 * kWave];                \
  V##3 = s[(base) + 3 * kWave]; V##4 = s[(base) + 4 * kWave]; V##5 = s[(base) + 5 * kWave];                \
  V##6 = s[(base) + 6 * kWave]; V##7 = s[(base) + 7 * kWave]; V##8 = s[(base) + 8 * kWave];                \
  V##9 = s[(base) + 9 * kWave]; V##10 = s[(base) + 10 * kWave]; V##11 = s[(base) + 11 * kWave];            \
  V##12 = s[(base) + 12 * kWave]; V##13 = s[(base) + 13 * kWave]; V##14 = s[(base) + 14 * kWave];          \
  V##15 = s[(base) + 15 * kWave];
#define MMA_STORE16(V, base)                                                                               \
  d[(base) + 0 * kWave] = V##0; d[(base) + 1 * kWave] = V##1; d[(base) + 2 * kWave] = V##2;                \
  d[(base) + 3 * kWave] = V##3; d[(base) + 4 * kWave] = V##4; d[(base) + 5 * kWave] = V##5;                \
  d[(base) + 6 * kWave] = V##6; d[(base) + 7 * kWave] = V##7; d[(base) + 8 * kWave] = V##8;                \
  d[(base) + 9 * kWave] = V##9; d[(base) + 10 * kWave] = V##10; d[(base) + 11 * kWave] = V##11;            \
  d[(base) + 12 * kWave] = V##12; d[(base) + 13 * kWave] = V##13; d[(base) + 14 * kWave] = V##14;          \
  d[(base) + 15 * kWave] = V##15;

// n16 16-byte units s[0, n16) -> d[0, n16), both aligned. Consecutive lanes
// move consecutive units, so each load instruction covers one contiguous 1 KiB
// span. Two register batches ping-pong: the loads of the next batch are issued
// before the current batch is stored, so a wave keeps up to 32 KiB of reads in
// flight.
__device__ __forceinline__ void aligned_units(const gu4* __restrict__ s0, gu4* __restrict__ d0, uint64_t n16,
                                              uint32_t lane) {
  const gu4* s = s0 + lane;  // this lane's unit
  gu4* d = d0 + lane;
  const uint64_t nb = n16 / kBatch;  // full batches (wave-uniform)
  if (nb > 0) {
    u32x4 a0, a1, a2, a3, a4, a5, a6, a7, a8, a9, a10, a11, a12, a13, a14, a15;
    u32x4 b0, b1, b2, b3, b4, b5, b6, b7, b8, b9, b10, b11, b12, b13, b14, b15;
    MMA_LOAD16(a, 0)
    uint64_t k = 0;  // batch held in registers `a` at the top of the loop
    for (;;) {
      if (k + 1 >= nb) {
        MMA_STORE16(a, k * kBatch)
        break;
      }
      MMA_LOAD16(b, (k + 1) * kBatch)
      __builtin_amdgcn_sched_barrier(0);
      MMA_STORE16(a, k * kBatch)
      ++k;
      if (k + 1 >= nb) {
        MMA_STORE16(b, k * kBatch)
        break;
      }
      MMA_LOAD16(a, (k + 1) * kBatch)
      __builtin_amdgcn_sched_barrier(0);
      MMA_STORE16(b, k * kBatch)
      ++k;
    }
  }
  // Remainder (< one batch): one batch, all loads issued before the first
  // store, so a short copy costs one round trip instead of one per 1 KiB. The
  // loads are unconditional -- a lane past the end re-reads the last unit -- and
  // only the stores are predicated: a predicated load makes the compiler wait
  // for it before the next one, one PCIe round trip each.
  const uint64_t r = nb * kBatch;
  if (r < n16) {
    const uint64_t left = n16 - r;  // units left for the whole wave, < kBatch
    u32x4 c0, c1, c2, c3, c4, c5, c6, c7, c8, c9, c10, c11, c12, c13, c14, c15;
#define MMA_PLD(k) c##k = s0[r + min(static_cast<uint64_t>((k) * kWave + lane), left - 1)];
#define MMA_PST(k) if ((k) * kWave + lane < left) d[r + (k) * kWave] = c##k;
    MMA_PLD(0) MMA_PLD(1) MMA_PLD(2) MMA_PLD(3) MMA_PLD(4) MMA_PLD(5) MMA_PLD(6) MMA_PLD(7)
    MMA_PLD(8) MMA_PLD(9) MMA_PLD(10) MMA_PLD(11) MMA_PLD(12) MMA_PLD(13) MMA_PLD(14) MMA_PLD(15)
    __builtin_amdgcn_sched_barrier(0);
    MMA_PST(0) MMA_PST(1) MMA_PST(2) MMA_PST(3) MMA_PST(4) MMA_PST(5) MMA_PST(6) MMA_PST(7)
    MMA_PST(8) MMA_PST(9) MMA_PST(10) MMA_PST(11) MMA_PST(12) MMA_PST(13) MMA_PST(14) MMA_PST(15)
#undef MMA_PLD
#undef MMA_PST
  }
}

// Bytes [4Q + r, 4Q + r + 16) of the 32 bytes lo|hi (little-endian), r < 4:
// v_alignbyte_b32 takes 4 bytes at a byte offset out of two adjacent words.
template <uint32_t Q>
__device__ __forceinline__ u32x4 funnel16(const u32x4& lo, const u32x4& hi, uint32_t r) {
  const uint32_t w[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  u32x4 o;
  o[0] = __builtin_amdgcn_alignbyte(w[Q + 1], w[Q], r);
  o[1] = __builtin_amdgcn_alignbyte(w[Q + 2], w[Q + 1], r);
  o[2] = __builtin_amdgcn_alignbyte(w[Q + 3], w[Q + 2], r);
  o[3] = __builtin_amdgcn_alignbyte(w[Q + 4], w[Q + 3], r);
  return o;
}

// One batch of a realigning copy: rows v[0..15] hold source units
// base + i * 64 + lane; `next` is unit base + kBatch, the same in every lane.
// A lane's unit k + 1 is its right neighbour's unit k (ds_bpermute); lane
// 63's is lane 0's of the next row (readlane), or `next` for the last row.
template <uint32_t Q>
__device__ __forceinline__ void realign_store(const u32x4 (&v)[16], const u32x4& next, gu4* __restrict__ d,
                                              uint64_t base, uint64_t n16, uint32_t r, uint32_t lane, int right) {
#pragma unroll
  for (uint32_t i = 0; i < 16; ++i) {
    u32x4 hi;
#pragma unroll
    for (uint32_t w = 0; w < 4; ++w) {
      const uint32_t nb = static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(right, static_cast<int>(v[i][w])));
      const uint32_t l0 = i < 15 ? __builtin_amdgcn_readlane(v[i + 1][w], 0) : next[w];
      hi[w] = lane == kWave - 1 ? l0 : nb;
    }
    const uint64_t u = base + i * kWave + lane;
    if (u < n16) d[u] = funnel16<Q>(v[i], hi, r);
  }
}

// n16 aligned destination units d[0, n16) from a source that starts
// s = 4Q + r bytes (1 <= s <= 15) past the aligned unit sa[0]: unit k is bytes
// [s, s + 16) of the aligned source units k and k + 1. Every load and store is
// an aligned 16-byte unit; the shift happens in registers. Source units
// [0, n16] each hold at least one byte of the source range, and loads past
// the end are clamped to unit n16, so no load leaves the aligned units the
// range touches; stores are predicated.
// kDeep = false: one 16 KiB batch in flight per wave; a batch's `next` unit is
// one more load that every lane makes at the same address (one request).
// kDeep = true: batches ping-pong as in aligned_units -- the next batch's loads
// are issued before this one is stored, and its first unit is this batch's
// `next` -- for 32 KiB in flight per wave; the last batch's `next`, unit n16,
// is read once at the start. It needs 64 more VGPRs, which only the lean
// self-contained kernel has to spare.
template <uint32_t Q, bool kDeep>
__device__ void realign_units(const gu4* __restrict__ sa, gu4* __restrict__ d, uint64_t n16, uint32_t r,
                              uint32_t lane) {
  const int right = static_cast<int>(((lane + 1) & (kWave - 1)) << 2);  // ds_bpermute byte address
  auto load = [&](u32x4 (&v)[16], uint64_t base) {
#pragma unroll
    for (uint32_t i = 0; i < 16; ++i) v[i] = sa[min(base + i * kWave + lane, n16)];
  };
  if constexpr (!kDeep) {
    for (uint64_t base = 0; base < n16; base += kBatch) {
      u32x4 v[16];
      load(v, base);
      const u32x4 next = sa[min(base + kBatch, n16)];
      __builtin_amdgcn_sched_barrier(0);
      realign_store<Q>(v, next, d, base, n16, r, lane, right);
    }
  } else {
    const u32x4 last = sa[n16];
    auto first = [&](const u32x4& v0) {
      u32x4 x;
#pragma unroll
      for (uint32_t w = 0; w < 4; ++w) x[w] = __builtin_amdgcn_readlane(v0[w], 0);
      return x;
    };
    u32x4 a[16], b[16];
    load(a, 0);
    for (uint64_t base = 0;;) {
      if (base + kBatch >= n16) {
        realign_store<Q>(a, last, d, base, n16, r, lane, right);
        break;
      }
      load(b, base + kBatch);
      __builtin_amdgcn_sched_barrier(0);
      realign_store<Q>(a, first(b[0]), d, base, n16, r, lane, right);
      base += kBatch;
      if (base + kBatch >= n16) {
        realign_store<Q>(b, last, d, base, n16, r, lane, right);
        break;
      }
      load(a, base + kBatch);
      __builtin_amdgcn_sched_barrier(0);
      realign_store<Q>(b, first(a[0]), d, base, n16, r, lane, right);
      base += kBatch;
    }
  }
}

// Wave-cooperative copy of n bytes. A byte head brings the destination to a
// 16-byte boundary; the aligned middle moves in 16-byte units -- straight
// (aligned_units) when source and destination are equally aligned modulo 16,
// else realigned in registers (realign_units); a byte tail finishes. The head
// and tail bytes are read first, with unconditional clamped loads, and
// written last, so their round trips overlap the middle's instead of
// preceding it. kDeep: see realign_units.
template <bool kDeep = false>
__device__ __forceinline__ void wave_copy(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
                                          uint64_t n, uint32_t lane) {
  const bool rel = ((reinterpret_cast<uintptr_t>(src) ^ reinterpret_cast<uintptr_t>(dst)) & 15u) != 0;
  uint64_t head = (16u - (reinterpret_cast<uintptr_t>(dst) & 15u)) & 15u;
  if (head > n) head = n;
  const uint64_t n16 = (n - head) >> 4, tail = (n - head) & 15u, tb = head + (n16 << 4);
  uint8_t hv = 0, tv = 0;
  if (head) hv = src[min(static_cast<uint64_t>(lane), head - 1)];
  if (tail) tv = src[tb + min(static_cast<uint64_t>(lane), tail - 1)];
  if (n16) {
    const uint8_t* s = src + head;
    gu4* d = (gu4*)(dst + head);
    if (!rel) {
      aligned_units((const gu4*)(s), d, n16, lane);
    } else {
      const uint32_t sh = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(s) & 15u);
      const gu4* sa = (const gu4*)(s - sh);
      switch (sh >> 2) {
        case 0: realign_units<0, kDeep>(sa, d, n16, sh & 3u, lane); break;
        case 1: realign_units<1, kDeep>(sa, d, n16, sh & 3u, lane); break;
        case 2: realign_units<2, kDeep>(sa, d, n16, sh & 3u, lane); break;
        default: realign_units<3, kDeep>(sa, d, n16, sh & 3u, lane); break;
      }
    }
  }
  if (lane < head) dst[lane] = hv;
  if (lane < tail) dst[tb + lane] = tv;
}

// ---------------------------------------------------------------- x-packed KV layout
// A paged-KV piece in the x-packed layout: key [H][R/16][B][16 bytes], value
// [H][D][B] elements, while the host keeps every piece token-major [B][H][R]
// (R = head_dim * elem bytes per token row of one head). Both transforms
// permute the piece at 16-byte (key) or element (value) granularity, so one
// side of a direct copy would be read or written in scattered 16-byte or
// smaller pieces -- across PCIe, requests that small waste most of each
// transaction. Each wave therefore stages a group of whole heads in its slice
// of LDS: it reads the group coalesced in the source's order, then writes it
// coalesced in the destination's order, gathering from LDS. Rows in LDS are
// padded by 16 bytes to spread the column reads over the banks.
typedef __attribute__((address_space(3))) uint8_t lds_u8;
typedef __attribute__((address_space(3))) u32x4 lu4;

// Make LDS writes of the wave visible to its other lanes (the wave-level
// barrier idiom: release, wave barrier, acquire).
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// 16-byte units [0, n) moved by one wave: map(u) gives the unit's source and
// destination offsets, get(source offset) reads it, put(destination offset, v)
// writes it. kUnits units per lane are read before the first is written; their
// offsets are computed once and kept in registers.
constexpr uint32_t kUnits = 8;
struct UnitOffs {
  uint32_t src, dst;
};
// Reads are unconditional (a lane past the end reads unit n - 1 again): a
// predicated read would make the compiler wait for it before issuing the next.
template <class Map, class Get, class Put>
__device__ __forceinline__ void wave_units(uint32_t n, uint32_t lane, Map map, Get get, Put put) {
  for (uint32_t base = 0; base < n; base += kUnits * kWave) {
    u32x4 v[kUnits];
    UnitOffs o[kUnits];
#pragma unroll
    for (uint32_t i = 0; i < kUnits; ++i) {
      o[i] = map(min(base + i * kWave + lane, n - 1));
      v[i] = get(o[i].src);
    }
#pragma unroll
    for (uint32_t i = 0; i < kUnits; ++i) {
      if (base + i * kWave + lane < n) put(o[i].dst, v[i]);
    }
  }
}

// 16 bytes made of 16 / E elements of E bytes, element j at p + j * stride (LDS).
template <uint32_t E>
__device__ __forceinline__ u32x4 gather16(const lds_u8* p, uint32_t stride) {
  u32x4 r;
  if constexpr (E == 1) {
#pragma unroll
    for (uint32_t w = 0; w < 4; ++w) {
      const lds_u8* q = p + 4 * w * stride;
      r[w] = static_cast<uint32_t>(q[0]) | (static_cast<uint32_t>(q[stride]) << 8) |
             (static_cast<uint32_t>(q[2 * stride]) << 16) | (static_cast<uint32_t>(q[3 * stride]) << 24);
    }
  } else if constexpr (E == 2) {
#pragma unroll
    for (uint32_t w = 0; w < 4; ++w) {
      const auto* q0 = reinterpret_cast<const __attribute__((address_space(3))) uint16_t*>(p + 2 * w * stride);
      const auto* q1 = reinterpret_cast<const __attribute__((address_space(3))) uint16_t*>(p + (2 * w + 1) * stride);
      r[w] = static_cast<uint32_t>(*q0) | (static_cast<uint32_t>(*q1) << 16);
    }
  } else if constexpr (E == 4) {
#pragma unroll
    for (uint32_t w = 0; w < 4; ++w) r[w] = *reinterpret_cast<const __attribute__((address_space(3))) uint32_t*>(p + w * stride);
  } else {
#pragma unroll
    for (uint32_t w = 0; w < 2; ++w) {
      const auto* q = reinterpret_cast<const __attribute__((address_space(3))) uint32_t*>(p + w * stride);
      r[2 * w] = q[0];
      r[2 * w + 1] = q[1];
    }
  }
  return r;
}

// host (token-major) piece `src` -> x-packed block `dst`; k = 0 key, 1 value.
template <uint32_t E>
__device__ void xpacked_to_block(const uint8_t* src, uint8_t* dst, uint32_t k, const XGeom& g, lds_u8* lds,
                                 uint32_t lane) {
  const uint32_t G = xp_to_heads(g);
  auto to_lds = [&](uint32_t o, u32x4 v) { *reinterpret_cast<lu4*>(lds + o) = v; };
  for (uint32_t h0 = 0; h0 < g.H; h0 += G) {
    const uint32_t gh = xp_min(G, g.H - h0), rs = xp_to_row_stride(g, gh);
    wave_units(xp_to_load_count(g, gh), lane,
               [&](uint32_t u) {
                 UnitOffs o;
                 xp_to_load(g, h0, gh, u, &o.src, &o.dst);
                 return o;
               },
               [&](uint32_t o) -> u32x4 { return *(const gu4*)(src + o); }, to_lds);
    wave_sync();
    uint8_t* out = dst + h0 * g.B * g.R;  // heads are the block's outermost dimension
    auto to_out = [&](uint32_t o, u32x4 v) { *(gu4*)(out + o) = v; };
    if (k == 0)
      wave_units(xp_to_key_count(g, gh), lane, [&](uint32_t v) { return UnitOffs{xp_to_key_lds(g, gh, v), v * 16}; },
                 [&](uint32_t o) -> u32x4 { return *reinterpret_cast<const lu4*>(lds + o); }, to_out);
    else
      wave_units(xp_to_val_count(g, gh), lane, [&](uint32_t v) { return UnitOffs{xp_to_val_lds(g, gh, v), v * 16}; },
                 [&](uint32_t o) -> u32x4 { return gather16<E>(lds + o, rs); }, to_out);
    wave_sync();  // the tile is read before the next group overwrites it
  }
}

// x-packed block `src` -> host (token-major) piece `dst`; k = 0 key, 1 value.
template <uint32_t E>
__device__ void xpacked_from_block(const uint8_t* src, uint8_t* dst, uint32_t k, const XGeom& g, lds_u8* lds,
                                   uint32_t lane) {
  const uint32_t G = xp_from_heads(g, k), rs = xp_from_row_stride(g, k);
  auto to_lds = [&](uint32_t o, u32x4 v) { *reinterpret_cast<lu4*>(lds + o) = v; };
  auto to_dst = [&](uint32_t o, u32x4 v) { *(gu4*)(dst + o) = v; };
  for (uint32_t h0 = 0; h0 < g.H; h0 += G) {
    const uint32_t gh = xp_min(G, g.H - h0);
    const uint8_t* in = src + h0 * g.B * g.R;  // the group is one contiguous range of the block
    wave_units(xp_from_load_count(g, k, gh), lane,
               [&](uint32_t v) { return UnitOffs{v * 16, xp_from_load_lds(g, k, v)}; },
               [&](uint32_t o) -> u32x4 { return *(const gu4*)(in + o); }, to_lds);
    wave_sync();
    if (k == 0)
      wave_units(xp_from_store_count(g, gh), lane,
                 [&](uint32_t u) { return UnitOffs{xp_from_store_lds(g, 0, gh, u), xp_from_store_dst(g, h0, gh, u)}; },
                 [&](uint32_t o) -> u32x4 { return *reinterpret_cast<const lu4*>(lds + o); }, to_dst);
    else
      wave_units(xp_from_store_count(g, gh), lane,
                 [&](uint32_t u) { return UnitOffs{xp_from_store_lds(g, 1, gh, u), xp_from_store_dst(g, h0, gh, u)}; },
                 [&](uint32_t o) -> u32x4 { return gather16<E>(lds + o, rs); }, to_dst);
    wave_sync();
  }
}

template <uint32_t E>
__device__ __forceinline__ void xpacked_piece(const uint8_t* src, uint8_t* dst, bool to_block, uint32_t k,
                                              const XGeom& g, lds_u8* lds, uint32_t lane) {
  if (to_block)
    xpacked_to_block<E>(src, dst, k, g, lds, lane);
  else
    xpacked_from_block<E>(src, dst, k, g, lds, lane);
}

// ---------------------------------------------------------------- head-major KV layout
// A paged-KV piece in the head-major (HND) layout: the block is [H][B][R], the
// host piece [B][H][R]. Whole rows move, so there is no LDS stage: units are
// taken in host order, which keeps the PCIe side (host reads of a fetch, host
// writes of an offload) contiguous, and the HBM side is read or written in whole
// rows (256 bytes for the 64k-token workload).
__device__ __forceinline__ void hnd_piece(const uint8_t* src, uint8_t* dst, bool to_block, const XGeom& g,
                                          uint32_t lane) {
  auto get = [&](uint32_t o) -> u32x4 { return *(const gu4*)(src + o); };
  auto put = [&](uint32_t o, u32x4 v) { *(gu4*)(dst + o) = v; };
  if (to_block)
    wave_units(hnd_count(g), lane, [&](uint32_t u) { return UnitOffs{u * 16, hnd_block_off(g, u)}; }, get, put);
  else
    wave_units(hnd_count(g), lane, [&](uint32_t u) { return UnitOffs{hnd_block_off(g, u), u * 16}; }, get, put);
}

// Template value of transfer_body for the head-major layout (the x-packed ones
// are the element sizes 1, 2, 4, 8).
constexpr uint32_t kXeHnd = 0x100;

extern __shared__ __attribute__((aligned(16))) uint8_t mma_dyn_lds[];

// The dummy-task kernel's body. kXE = 0: paged-KV blocks hold pieces as the
// host does. kXE = kXeHnd: head-major blocks (a row permutation, no LDS).
// kXE = element bytes: the x-packed GPU block layout through LDS --
// one kernel per element size, so that no launch carries the registers or LDS
// of a transform it does not run.
template <uint32_t kXE>
__device__ __forceinline__ void transfer_body(const KernelArgs& a) {
  __shared__ uint64_t s_layer[kMaxLayers];
  Record* rec = a.rec;
  DevState* ds = a.ds;
  const uint32_t lane = threadIdx.x & (kWave - 1);

  // KV layer table from the kernel arguments into LDS.
  const uint32_t nl = a.kv_layers < kMaxLayers ? a.kv_layers : kMaxLayers;
  for (uint32_t i = threadIdx.x; i < nl; i += kBlock) s_layer[i] = a.layer_ptr[i];
  const uint64_t piece = a.kv_piece_bytes;
  const uint64_t kstride = a.kv_kstride;
  const XGeom xg{a.kv_tokens, a.kv_heads, a.kv_row_bytes, a.kv_elem, a.kv_lds_wave};
  lds_u8* wave_lds = (lds_u8*)(mma_dyn_lds) + (threadIdx.x / kWave) * a.kv_lds_wave;
  __syncthreads();

  // One ring entry: words a, b and count | kind_p0 (see CuEntry). One copy site
  // for every kind (a linear entry is a single "piece"), so the copy loop is
  // instantiated once.
  auto run_entry = [&](uint64_t w1, uint64_t w2, uint64_t w3) {
    const uint32_t count = static_cast<uint32_t>(w3);
    const uint32_t kind = static_cast<uint32_t>(w3 >> 32) & kEntryKindMask;
    const uint32_t p0 = static_cast<uint32_t>(w3 >> 40);
    // Data landed by an SDMA engine during this kernel: drop any stale copy of
    // it from this CU's vector L1 (and non-coherent L2 lines) before reading.
    if ((w3 >> 32) & kEntryAcquire) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");
    const bool paged = kind != kEntryCopy;
    const uint32_t npieces = paged ? count : 1u;
    for (uint32_t j = 0; j < npieces; ++j) {
      const uint8_t* src = reinterpret_cast<const uint8_t*>(w1);
      uint8_t* dst = reinterpret_cast<uint8_t*>(w2);
      uint64_t n = count;
      if (paged) {
        const uint32_t p = p0 + j;
        uint8_t* pg = reinterpret_cast<uint8_t*>(s_layer[p >> 1]) + (p & 1u) * kstride + w2 * piece;
        uint8_t* contig = reinterpret_cast<uint8_t*>(w1) + j * piece;
        src = kind == kEntryToPaged ? contig : pg;
        dst = kind == kEntryToPaged ? pg : contig;
        n = piece;
        if constexpr (kXE == kXeHnd) {
          hnd_piece(src, dst, kind == kEntryToPaged, xg, lane);
          continue;
        } else if constexpr (kXE != 0) {
          xpacked_piece<kXE>(src, dst, kind == kEntryToPaged, p & 1u, xg, wave_lds, lane);
          continue;
        }
      }
      wave_copy(src, dst, n, lane);
    }
  };

  // A self-contained launch of a whole KV transfer (linear ones use
  // mma_whole_kernel): wave w copies entry w of the arguments and writes its
  // done tag -- no start signal, record, ring or wait.
  if (a.self_contained) {
    const uint32_t w = blockIdx.x * kWavesPerWG + threadIdx.x / kWave;
    if (w < a.n_pre) {
      run_entry(a.pre[w][0], a.pre[w][1], a.pre[w][2]);
      if (a.release_each) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "");
      if (lane == 0) st_sys(&a.done[w], make_tag(a.seq, w));
    }
    return;
  }

  // 1. start signal (stream -> engine). Work that precedes this kernel in
  // stream order is complete and visible (dispatch acquire/release).
  if (lane == 0) {
    const uint32_t first = __hip_atomic_fetch_add(&ds->arrived, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (first == 0) st_sys(&rec->h.started, a.seq);
  }

  // 2. CU-path worker loop. Lane 0 claims; lanes 0..4 fetch the entry with one
  // load instruction; the wave copies.
  uint64_t hb = 0, t_prog = 0;
  uint32_t timed_out = 0;
  if (lane == 0) t_prog = wall_clock64();
  for (;;) {
    uint64_t x = 0;
    if (lane == 0)
      x = __hip_atomic_fetch_add(&ds->cursor, static_cast<uint64_t>(1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    x = lane_u64(x, 0);
    if (a.device_ctl && x >= a.n_total) break;  // the whole CU share was in the ring at launch
    const uint64_t expect = make_tag(a.seq, x);
    const uint64_t* ew = reinterpret_cast<const uint64_t*>(&rec->ring[x % kRingSize]);
    uint32_t state = 0;  // 1: entry ready, 3: watchdog
    uint64_t w1 = 0, w2 = 0, w3 = 0;
    if (x < a.n_pre) {  // first entries arrive with the launch: no PCIe round trip
      w1 = a.pre[x][0];
      w2 = a.pre[x][1];
      w3 = a.pre[x][2];
      state = 1;
    }
    for (uint32_t polls = 0; state == 0; ++polls) {
      const uint64_t w = lane < 5 ? ld_sys(ew + lane) : 0;
      if (lane_u64(w, 0) == expect && lane_u64(w, 4) == expect) {
        w1 = lane_u64(w, 1);
        w2 = lane_u64(w, 2);
        w3 = lane_u64(w, 3);
        state = 1;
        break;
      }
      if ((polls & 7) == 7) {  // watchdog check every 8th poll
        uint32_t st = 0;
        if (lane == 0) {
          const uint64_t now = wall_clock64();
          const uint64_t hb2 = ld_sys(&rec->h.heartbeat);
          if (hb2 != hb) {
            hb = hb2;
            t_prog = now;
          } else if (now - t_prog > a.watchdog_ticks ||
                     __hip_atomic_load(&ds->timed_out, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) {
            st = 3;
          }
        }
        st = __builtin_amdgcn_readfirstlane(st);
        if (st) {
          state = st;
          break;
        }
      }
      backoff(polls < 4 ? 1u : (polls < 16 ? 4u : 8u));
    }
    if (state != 1) {
      if (state == 3) timed_out = 1;
      break;
    }
    if ((static_cast<uint32_t>(w3 >> 32) & kEntryKindMask) == kEntryEnd)
      break;  // the ring is closed and this ticket is past its end
    run_entry(w1, w2, w3);
    if (a.release_each) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "");
    if (lane == 0) {
      st_sys(&a.done[x % kRingSize], expect);
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
      int32_t status = 0;
      if (a.device_ctl) {
        // Every wave has left, so the CU share has landed; the copy engines'
        // share has when their completion signal reaches 0. Nothing re-arms
        // the watchdog here: it runs from this wave's last completion.
        int64_t left = 0;
        while (!to && a.sdma_left &&
               (left = __hip_atomic_load(const_cast<int64_t*>(a.sdma_left), __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_SYSTEM)) > 0) {
          if (wall_clock64() - t_prog > a.watchdog_ticks) to = 1;
          __builtin_amdgcn_s_sleep(8);
        }
        if (left < 0) status = 2;
      } else {
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
      }
      if (to) status = 1;
      if (status) __hip_atomic_store(&rec->h.status, status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      __hip_atomic_store(&ds->cursor, static_cast<uint64_t>(0), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&ds->arrived, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&ds->exited, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&ds->timed_out, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "");
      st_sys(&rec->h.released, a.seq);
    }
  }
}

}  // namespace

__global__ __launch_bounds__(kBlock) void mma_transfer_kernel(KernelArgs a) { transfer_body<0>(a); }

// A self-contained launch: every entry of a linear transfer travels in the
// arguments and no copy engine takes part, so wave w of the grid copies entry w
// and writes its done tag -- no start signal, ring, exit count or wait. The
// arguments hold only the entries (N of them), so a deep queue of small
// transfers on one stream uses little of the runtime's kernel-argument pool.
template <uint32_t N>
__global__ __launch_bounds__(kBlock) void mma_whole_kernel(WholeArgs<N> a) {
  const uint32_t lane = threadIdx.x & (kWave - 1);
  const uint32_t w = blockIdx.x * kWavesPerWG + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  if (w >= a.n) return;
  wave_copy<true>(reinterpret_cast<const uint8_t*>(a.e[w][0]), reinterpret_cast<uint8_t*>(a.e[w][1]),
                  static_cast<uint32_t>(a.e[w][2]), lane);
  if (a.release_each) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "");
  if (lane == 0) st_sys(&a.done[w], make_tag(a.seq, w));
}

__global__ __launch_bounds__(kBlock) void mma_transfer_hnd_kernel(KernelArgs a) { transfer_body<kXeHnd>(a); }

// One span of an HBM pool launch: n <= kPoolSpan bytes. A full, 16-byte
// aligned span is read whole into registers before the first store, with
// nontemporal loads and stores (every byte is moved once, so caching it would
// only evict other data); a piece's shorter last span and misaligned spans
// take plain loops.
constexpr uint32_t kPoolVec = kPoolSpan / (kWave * 16);
__device__ __forceinline__ void pool_span(const uint8_t* src, uint8_t* dst, uint32_t n, uint32_t lane) {
  const uintptr_t mis = (reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) & 15u;
  if (mis == 0 && n == kPoolSpan) {
    const gu4* s = (const gu4*)(src) + lane;
    gu4* d = (gu4*)(dst) + lane;
    u32x4 v[kPoolVec];
#pragma unroll
    for (uint32_t i = 0; i < kPoolVec; ++i) v[i] = __builtin_nontemporal_load(s + i * kWave);
#pragma unroll
    for (uint32_t i = 0; i < kPoolVec; ++i) __builtin_nontemporal_store(v[i], d + i * kWave);
    return;
  }
  if (mis == 0) {
    const uint32_t n16 = n >> 4;
    const gu4* s = (const gu4*)(src);
    gu4* d = (gu4*)(dst);
    for (uint32_t i = lane; i < n16; i += kWave) d[i] = s[i];
    for (uint32_t i = (n16 << 4) + lane; i < n; i += kWave) dst[i] = src[i];
    return;
  }
  for (uint32_t i = lane; i < n; i += kWave) dst[i] = src[i];
}

// A paged-KV transfer between a pool in this GPU's memory and the paged layer
// tensors (piece layout): HBM-bound, so the launch is sized to the bytes, up
// to kPoolMaxWorkgroups workgroups, with no ring and no host round trip. A
// workgroup's spans are contiguous and its waves interleave over them, so a
// wave meets one or two blocks and reads each one's table entry once. The
// counter only orders the done tag after every workgroup has finished with its
// table entries: the data itself becomes visible to later work through the
// stream, when the kernel ends, as for any kernel (a device-wide release per
// workgroup would write back the L2 of its XCD each time).
// kHnd: GPU blocks in the head-major layout; a span is then a whole piece,
// permuted row by row on its way (hnd_piece).
template <bool kHnd>
__global__ __launch_bounds__(kBlock) void mma_kv_pool_kernel(PoolArgs a) {
  const uint32_t lane = threadIdx.x & (kWave - 1);
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const uint64_t u0 = static_cast<uint64_t>(blockIdx.x) * a.per_wg;
  const uint64_t u1 = min(a.units, u0 + a.per_wg);
  const uint64_t per_blk = static_cast<uint64_t>(a.ppb) * a.spans;
  uint64_t cur = ~0ull, pooled = 0, paged_off = 0;
  for (uint64_t u = u0 + wave; u < u1; u += kWavesPerWG) {
    const uint64_t i = u / per_blk;
    const uint32_t r = static_cast<uint32_t>(u - i * per_blk);
    const uint32_t p = r / a.spans;
    const uint32_t sp = r - p * a.spans;
    if (i != cur) {
      cur = i;
      const uint64_t e = ld_sys(&a.tab[i]);
      pooled = a.pool + (e & 0xffffffffull) * a.slot_bytes;
      paged_off = (e >> 32) * a.piece;
    }
    const uint64_t off = static_cast<uint64_t>(sp) * kPoolSpan;
    const uint32_t n = static_cast<uint32_t>(min(static_cast<uint64_t>(kPoolSpan), a.piece - off));
    uint8_t* host_side = reinterpret_cast<uint8_t*>(pooled + static_cast<uint64_t>(p) * a.piece + off);
    uint8_t* gpu_side = reinterpret_cast<uint8_t*>(a.layer_ptr[p >> 1] + (p & 1u) * a.kstride + paged_off + off);
    if constexpr (kHnd) {
      const XGeom g{a.tokens, a.heads, a.row_bytes, a.elem, 0};
      if (a.to_paged)
        hnd_piece(host_side, gpu_side, true, g, lane);
      else
        hnd_piece(gpu_side, host_side, false, g, lane);
    } else if (a.to_paged)
      pool_span(host_side, gpu_side, n, lane);
    else
      pool_span(gpu_side, host_side, n, lane);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t prev = __hip_atomic_fetch_add(a.ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (prev == gridDim.x - 1) {
      __hip_atomic_store(a.ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
      st_sys(a.done, make_tag(a.seq, 0));
    }
  }
}

template <uint32_t E>
__global__ __launch_bounds__(kBlock) void mma_transfer_xpacked_kernel(KernelArgs a) {
  transfer_body<E>(a);
}

// ------------------------------------------------------- KV fetch that allocates nothing
// Table chunk of a no-alloc KV fetch: entries [first, first + count) of the
// call's block table from the arguments into the scratch array; the first
// chunk of a call also returns the claim counter to 0.
__global__ __launch_bounds__(kBlock) void mma_kv_noalloc_table_kernel(NoallocTabArgs a) {
  uint64_t* tab = a.scratch + kNoallocTabOffset / 8;
  for (uint32_t j = threadIdx.x; j < a.count; j += kBlock) tab[a.first + j] = a.e[j];
  if (a.reset && threadIdx.x == 0) a.scratch[0] = 0;
}

// The pieces of a no-alloc KV fetch, carried by the CU path alone: a wave
// claims per_claim consecutive pieces (piece u is piece u % ppb of table entry
// u / ppb) from the counter in the scratch array, looks up their block, and
// copies host slot -> paged layer in the GPU block layout of kXE (as for
// transfer_body: 0 pieces as on the host, kXeHnd head-major, else the x-packed
// element size). No ring, no record, no host thread: the data is complete
// when the kernel ends, and the stream orders it for later work.
template <uint32_t kXE>
__global__ __launch_bounds__(kBlock) void mma_kv_noalloc_kernel(NoallocArgs a) {
  const uint32_t lane = threadIdx.x & (kWave - 1);
  const XGeom xg{a.tokens, a.heads, a.row_bytes, a.elem, a.lds_wave};
  lds_u8* wave_lds = (lds_u8*)(mma_dyn_lds) + (threadIdx.x / kWave) * a.lds_wave;
  const uint64_t* tab = a.scratch + kNoallocTabOffset / 8;
  for (;;) {
    uint64_t c = 0;
    if (lane == 0)
      c = __hip_atomic_fetch_add(a.scratch, static_cast<uint64_t>(1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    c = lane_u64(c, 0);
    const uint64_t u0 = c * a.per_claim;
    if (u0 >= a.units) break;
    const uint64_t u1 = min(u0 + a.per_claim, a.units);
    for (uint64_t u = u0; u < u1; ++u) {
      const uint64_t i = u / a.ppb;
      const uint32_t p = static_cast<uint32_t>(u - i * a.ppb);
      const uint64_t e = lane_u64(tab[i], 0);
      const uint8_t* src = reinterpret_cast<const uint8_t*>(a.pool + (e & 0xffffffffull) * a.slot_bytes + p * a.piece);
      uint8_t* dst = reinterpret_cast<uint8_t*>(a.layer_ptr[p >> 1] + (p & 1u) * a.kstride + (e >> 32) * a.piece);
      if constexpr (kXE == kXeHnd)
        hnd_piece(src, dst, true, xg, lane);
      else if constexpr (kXE != 0)
        xpacked_piece<kXE>(src, dst, true, p & 1u, xg, wave_lds, lane);
      else
        wave_copy(src, dst, a.piece, lane);
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

template <uint32_t N>
hipError_t launch_whole(const KernelArgs& args, uint32_t grid, hipStream_t stream) {
  WholeArgs<N> w;
  w.done = args.done;
  w.seq = args.seq;
  w.n = args.n_pre;
  w.release_each = args.release_each;
  for (uint32_t i = 0; i < args.n_pre; ++i)
    for (int k = 0; k < 3; ++k) w.e[i][k] = args.pre[i][k];
  void* params[] = {&w};
  return hipLaunchKernel(reinterpret_cast<const void*>(&mma_whole_kernel<N>), dim3(grid), dim3(kBlock), params, 0,
                         stream);
}

hipError_t launch_pool(const KernelArgs& args, uint32_t grid, hipStream_t stream) {
  PoolArgs p;
  p.done = args.done;
  p.seq = args.seq;
  p.ctr = args.pool_ctr;
  p.tab = args.pool_tab;
  p.pool = args.pool_base;
  p.units = args.pool_units;
  p.per_wg = args.pool_per_wg;
  p.ppb = 2 * args.kv_layers;
  p.piece = args.kv_piece_bytes;
  p.slot_bytes = p.piece * p.ppb;
  p.kstride = args.kv_kstride;
  p.spans = args.pool_spans;
  p.to_paged = args.pool_to_paged;
  p.layers = args.kv_layers;
  p.tokens = args.kv_tokens;
  p.heads = args.kv_heads;
  p.row_bytes = args.kv_row_bytes;
  p.elem = args.kv_elem;
  for (uint32_t l = 0; l < args.kv_layers; ++l) p.layer_ptr[l] = args.layer_ptr[l];
  void* params[] = {&p};
  const void* k = args.kv_layout == kKvLayoutHnd ? reinterpret_cast<const void*>(&mma_kv_pool_kernel<true>)
                                                 : reinterpret_cast<const void*>(&mma_kv_pool_kernel<false>);
  return hipLaunchKernel(k, dim3(grid), dim3(kBlock), params, 0, stream);
}

hipError_t launch_transfer(const KernelArgs& args, uint32_t grid, hipStream_t stream) {
  if (args.pool_tab) return launch_pool(args, grid, stream);
  if (args.self_contained && args.kv_layers == 0) {  // linear: the lean kernel; KV: below, by layout
    if (args.n_pre <= 4) return launch_whole<4>(args, grid, stream);
    if (args.n_pre <= 16) return launch_whole<16>(args, grid, stream);
    return launch_whole<kPrefill>(args, grid, stream);
  }
  void* params[] = {const_cast<KernelArgs*>(&args)};
  // Only x-packed KV transfers stage through LDS; every other launch asks for
  // none, so it can share CUs with kernels that use most of theirs.
  if (args.kv_layout == kKvLayoutXPacked) {
    const void* k = args.kv_elem == 1   ? reinterpret_cast<const void*>(&mma_transfer_xpacked_kernel<1>)
                    : args.kv_elem == 2 ? reinterpret_cast<const void*>(&mma_transfer_xpacked_kernel<2>)
                    : args.kv_elem == 4 ? reinterpret_cast<const void*>(&mma_transfer_xpacked_kernel<4>)
                                        : reinterpret_cast<const void*>(&mma_transfer_xpacked_kernel<8>);
    return hipLaunchKernel(k, dim3(grid), dim3(kBlock), params, kWavesPerWG * args.kv_lds_wave, stream);
  }
  if (args.kv_layout == kKvLayoutHnd)
    return hipLaunchKernel(reinterpret_cast<const void*>(&mma_transfer_hnd_kernel), dim3(grid), dim3(kBlock), params,
                           0, stream);
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


// ------------------------------------------------------- KV fetch that allocates nothing
// The no-alloc KV fetch's claim counter and block table: a fixed array of this
// library's device code, so that the call needs no allocation. Every GPU the
// library runs on holds its own copy, at its own address, until the process
// ends. In host code the array's name is only a stand-in: its device address
// is looked up once per device (noalloc_setup, called by mma_init with that
// device current) and only that address is used.
static __device__ __align__(256) uint8_t scratch[kNoallocScratchBytes];

namespace {
constexpr int kNoallocDevices = 64;
uint64_t* g_scratch_dev[kNoallocDevices] = {};
}  // namespace

hipError_t noalloc_setup(int dev) {
  if (dev < 0 || dev >= kNoallocDevices) return hipErrorInvalidDevice;
  if (g_scratch_dev[dev]) return hipSuccess;
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  if (!p || (reinterpret_cast<uintptr_t>(p) & 255u) != 0) return hipErrorInvalidSymbol;
  g_scratch_dev[dev] = static_cast<uint64_t*>(p);
  return hipSuccess;
}

uint64_t* noalloc_scratch(int dev) { return dev >= 0 && dev < kNoallocDevices ? g_scratch_dev[dev] : nullptr; }

hipError_t launch_noalloc_table(const NoallocTabArgs& t, hipStream_t stream) {
  void* params[] = {const_cast<NoallocTabArgs*>(&t)};
  return hipLaunchKernel(reinterpret_cast<const void*>(&mma_kv_noalloc_table_kernel), dim3(1), dim3(kBlock), params,
                         0, stream);
}

hipError_t launch_noalloc(const NoallocArgs& a, uint32_t grid, hipStream_t stream) {
  void* params[] = {const_cast<NoallocArgs*>(&a)};
  const void* k = reinterpret_cast<const void*>(&mma_kv_noalloc_kernel<0>);
  uint32_t lds = 0;
  if (a.layout == kKvLayoutHnd) {
    k = reinterpret_cast<const void*>(&mma_kv_noalloc_kernel<kXeHnd>);
  } else if (a.layout == kKvLayoutXPacked) {
    k = a.elem == 1   ? reinterpret_cast<const void*>(&mma_kv_noalloc_kernel<1>)
        : a.elem == 2 ? reinterpret_cast<const void*>(&mma_kv_noalloc_kernel<2>)
        : a.elem == 4 ? reinterpret_cast<const void*>(&mma_kv_noalloc_kernel<4>)
                      : reinterpret_cast<const void*>(&mma_kv_noalloc_kernel<8>);
    lds = kWavesPerWG * a.lds_wave;
  }
  return hipLaunchKernel(k, dim3(grid), dim3(kBlock), params, lds, stream);
}

}  // namespace mma
