// CPU emulation of one wave running the dummy-task kernel's copy of a range
// whose ends differ in alignment modulo 16 (wave_copy / realign_units in
// mma_kernels.hip): a byte head to align the destination, aligned 16-byte
// source units shifted into aligned destination units in registers -- the
// right neighbour's unit through ds_bpermute, lane 0 of the next row through
// readlane -- and a byte tail.
//
// Lanes are emulated explicitly, with the kernel's batch shape (16 rows of 64
// lanes), both of its batch schedules (one batch in flight with a `next` unit
// loaded per batch; two batches ping-ponging, the next batch's first unit
// taken by readlane), its clamped loads and predicated stores, its head and
// tail bytes read first and written last, and v_alignbyte_b32's definition.
// Every load is checked to stay inside the aligned 16-byte units
// that the source range touches, every store inside the destination range,
// and every destination byte must be written exactly once; the result must
// equal the source. Run by tests/test_realign_emu.py over sizes and all 16 x 16
// alignment pairs (the relatively aligned ones are skipped: another path).
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

namespace {

constexpr uint32_t kWave = 64;
constexpr uint64_t kBatch = 16 * kWave;  // 16-byte units per batch

struct U4 {
  uint32_t w[4];
};

// v_alignbyte_b32 D = ({hi, lo} >> (8 * (sel & 3)))[31:0]
uint32_t alignbyte(uint32_t hi, uint32_t lo, uint32_t sel) {
  const uint64_t x = (static_cast<uint64_t>(hi) << 32) | lo;
  return static_cast<uint32_t>(x >> (8 * (sel & 3)));
}

U4 funnel16(const U4& lo, const U4& hi, uint32_t q, uint32_t r) {
  const uint32_t w[8] = {lo.w[0], lo.w[1], lo.w[2], lo.w[3], hi.w[0], hi.w[1], hi.w[2], hi.w[3]};
  U4 o;
  for (uint32_t j = 0; j < 4; ++j) o.w[j] = alignbyte(w[q + j + 1], w[q + j], r);
  return o;
}

struct Mem {
  // Source and destination live in separate arenas with guard bytes around the
  // ranges; accesses are checked before they are made.
  std::vector<uint8_t> src_arena, dst_arena;
  uint64_t src_off = 0, dst_off = 0, n = 0;
  std::vector<uint8_t> writes;
  int bad = 0;

  // a 16-byte aligned unit of the source arena at byte offset `off`
  U4 load_unit(uint64_t off) {
    const uint64_t lo = src_off & ~15ull, hi = (src_off + n + 15) & ~15ull;  // units the range touches
    if (off % 16 || off < lo || off + 16 > hi) {
      if (!bad) bad = 1;
      return U4{{0, 0, 0, 0}};
    }
    U4 v;
    memcpy(v.w, &src_arena[off], 16);
    return v;
  }
  uint8_t load_byte(uint64_t off) {
    if (off < src_off || off >= src_off + n) {
      if (!bad) bad = 2;
      return 0;
    }
    return src_arena[off];
  }
  void store_unit(uint64_t off, const U4& v) {
    if (off % 16 || off < dst_off || off + 16 > dst_off + n) {
      if (!bad) bad = 3;
      return;
    }
    memcpy(&dst_arena[off], v.w, 16);
    for (uint64_t b = 0; b < 16; ++b) ++writes[off - dst_off + b];
  }
  void store_byte(uint64_t off, uint8_t v) {
    if (off < dst_off || off >= dst_off + n) {
      if (!bad) bad = 4;
      return;
    }
    dst_arena[off] = v;
    ++writes[off - dst_off];
  }
};

// Offsets are arena offsets; the arenas are 16-byte aligned, so an offset's
// alignment is the address's.
void realign_store(Mem& m, const std::vector<U4>& v, const U4& next, uint64_t d, uint64_t base, uint64_t n16,
                   uint32_t q, uint32_t r) {
  for (uint32_t i = 0; i < 16; ++i) {
    U4 hi[kWave];
    for (uint32_t lane = 0; lane < kWave; ++lane) {
      const uint32_t right = (lane + 1) & (kWave - 1);          // ds_bpermute source lane
      const U4 nb = v[i * kWave + right];
      const U4 l0 = i < 15 ? v[(i + 1) * kWave + 0] : next;     // readlane(row i + 1, 0) / next
      hi[lane] = lane == kWave - 1 ? l0 : nb;
    }
    for (uint32_t lane = 0; lane < kWave; ++lane) {
      const uint64_t u = base + i * kWave + lane;
      if (u < n16) m.store_unit(d + 16 * u, funnel16(v[i * kWave + lane], hi[lane], q, r));
    }
  }
}

std::vector<U4> load_batch(Mem& m, uint64_t sa, uint64_t base, uint64_t n16) {
  std::vector<U4> v(16 * kWave);  // v[i * 64 + lane]
  for (uint32_t i = 0; i < 16; ++i)
    for (uint32_t lane = 0; lane < kWave; ++lane)
      v[i * kWave + lane] = m.load_unit(sa + 16 * std::min<uint64_t>(base + i * kWave + lane, n16));
  return v;
}

void realign_units(Mem& m, uint64_t sa, uint64_t d, uint64_t n16, uint32_t q, uint32_t r, bool deep) {
  if (!deep) {
    for (uint64_t base = 0; base < n16; base += kBatch) {
      const std::vector<U4> v = load_batch(m, sa, base, n16);
      const U4 next = m.load_unit(sa + 16 * std::min<uint64_t>(base + kBatch, n16));  // same address in every lane
      realign_store(m, v, next, d, base, n16, q, r);
    }
    return;
  }
  // ping-pong: the next batch is loaded before this one is stored; its row 0,
  // lane 0 (readlane) is this batch's `next`; the last batch's is unit n16
  const U4 last = m.load_unit(sa + 16 * n16);
  std::vector<U4> cur = load_batch(m, sa, 0, n16);
  for (uint64_t base = 0;; base += kBatch) {
    if (base + kBatch >= n16) {
      realign_store(m, cur, last, d, base, n16, q, r);
      break;
    }
    std::vector<U4> nxt = load_batch(m, sa, base + kBatch, n16);
    realign_store(m, cur, nxt[0], d, base, n16, q, r);
    cur.swap(nxt);
  }
}

// The kernel's wave_copy for a relatively misaligned range: head and tail
// bytes read first (unconditional loads, clamped into the range), the aligned
// middle realigned, head and tail written last.
void wave_copy_realign(Mem& m, uint64_t src, uint64_t dst, uint64_t n, bool deep) {
  uint64_t head = (16u - (dst & 15u)) & 15u;
  if (head > n) head = n;
  const uint64_t n16 = (n - head) >> 4, tail = (n - head) & 15u, tb = head + (n16 << 4);
  uint8_t hv[kWave] = {}, tv[kWave] = {};
  for (uint32_t lane = 0; lane < kWave; ++lane) {
    if (head) hv[lane] = m.load_byte(src + std::min<uint64_t>(lane, head - 1));
    if (tail) tv[lane] = m.load_byte(src + tb + std::min<uint64_t>(lane, tail - 1));
  }
  if (n16) {
    const uint64_t s = src + head, sh = s & 15u;
    realign_units(m, s - sh, dst + head, n16, static_cast<uint32_t>(sh >> 2), static_cast<uint32_t>(sh & 3u), deep);
  }
  for (uint32_t lane = 0; lane < kWave; ++lane) {
    if (lane < head) m.store_byte(dst + lane, hv[lane]);
    if (lane < tail) m.store_byte(dst + tb + lane, tv[lane]);
  }
}

// 0 on success; otherwise a code naming the first failure.
int check(uint64_t n, uint32_t so, uint32_t dof, uint32_t seed, bool deep) {
  Mem m;
  const uint64_t guard = 64;
  m.src_off = guard + so;
  m.dst_off = guard + dof;
  m.n = n;
  m.src_arena.resize(n + 2 * guard + 32);
  m.dst_arena.assign(n + 2 * guard + 32, 0xEE);
  m.writes.assign(n, 0);
  uint32_t x = seed * 2654435761u + 1;
  for (auto& b : m.src_arena) {
    x ^= x << 13;
    x ^= x >> 17;
    x ^= x << 5;
    b = static_cast<uint8_t>(x);
  }
  wave_copy_realign(m, m.src_off, m.dst_off, n, deep);
  if (m.bad) return 10 + m.bad;
  for (uint64_t i = 0; i < n; ++i)
    if (m.writes[i] != 1) return 20;
  if (memcmp(&m.dst_arena[m.dst_off], &m.src_arena[m.src_off], n) != 0) return 30;
  for (uint64_t i = 0; i < m.dst_arena.size(); ++i)
    if ((i < m.dst_off || i >= m.dst_off + n) && m.dst_arena[i] != 0xEE) return 40;
  return 0;
}

}  // namespace

// Usage: realign_emu n_max step [big sizes...]: every size 0..n_max in steps of `step`, and the
// given sizes, at every relatively misaligned (source, destination) offset pair modulo 16.
int main(int argc, char** argv) {
  if (argc < 3) return 2;
  const uint64_t n_max = strtoull(argv[1], nullptr, 0), step = strtoull(argv[2], nullptr, 0);
  std::vector<uint64_t> sizes;
  for (uint64_t n = 0; n <= n_max; n += step) sizes.push_back(n);
  for (int i = 3; i < argc; ++i) sizes.push_back(strtoull(argv[i], nullptr, 0));
  uint64_t cases = 0;
  for (uint64_t n : sizes)
    for (uint32_t so = 0; so < 16; ++so)
      for (uint32_t dof = 0; dof < 16; ++dof) {
        if (so == dof) continue;
        for (int deep = 0; deep < 2; ++deep) {
          const int rc = check(n, so, dof, static_cast<uint32_t>(n * 256 + so * 16 + dof), deep != 0);
          if (rc) {
            printf("FAIL n=%llu src+%u dst+%u deep=%d code=%d\n", static_cast<unsigned long long>(n), so, dof, deep,
                   rc);
            return 1;
          }
          ++cases;
        }
      }
  printf("ok %llu cases\n", static_cast<unsigned long long>(cases));
  return 0;
}
