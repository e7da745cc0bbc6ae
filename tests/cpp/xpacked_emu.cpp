// CPU emulation of one wave running the x-packed KV transform of the dummy-task
// kernel, over the same index maps (paper_2512_16056_amd/csrc/mma_xpacked.h):
// head groups, a load phase into the wave's LDS tile, a store phase out of it,
// value units gathered element by element at the tile's row stride. Every global
// access is checked against the piece, every LDS access against the tile
// capacity, and every destination byte must be written exactly once. Built into
// a small shared library by tests/test_xpacked_index.py and compared there with
// the oracle.
#include <cstdint>
#include <cstring>
#include <vector>

#include "mma_xpacked.h"

using namespace mma;

extern "C" int emu_xpacked(const uint8_t* src, uint8_t* dst, int to_block, int k, uint32_t B, uint32_t H, uint32_t R,
                           uint32_t E, uint32_t cap) {
  const XGeom g{B, H, R, E, cap};
  const uint64_t piece = static_cast<uint64_t>(B) * H * R;
  std::vector<uint8_t> lds(cap, 0xCD);
  std::vector<uint8_t> written(piece, 0);
  int bad = 0;
  auto gl = [&](uint64_t off, uint64_t len) {
    if (off + len > piece) bad = bad ? bad : 1;
    return off + len <= piece;
  };
  auto lo = [&](uint64_t off, uint64_t len) {
    if (off + len > cap) bad = bad ? bad : 2;
    return off + len <= cap;
  };
  auto put = [&](uint64_t off, const uint8_t* p, uint64_t len) {
    if (!gl(off, len)) return;
    std::memcpy(dst + off, p, len);
    for (uint64_t i = 0; i < len; ++i) written[off + i] += 1;
  };
  if (to_block) {
    const uint32_t G = xp_to_heads(g);
    for (uint32_t h0 = 0; h0 < H; h0 += G) {
      const uint32_t gh = xp_min(G, H - h0), rs = xp_to_row_stride(g, gh);
      for (uint32_t u = 0; u < xp_to_load_count(g, gh); ++u) {
        uint32_t so, l;
        xp_to_load(g, h0, gh, u, &so, &l);
        if (gl(so, 16) && lo(l, 16)) std::memcpy(&lds[l], src + so, 16);
      }
      const uint64_t out = static_cast<uint64_t>(h0) * B * R;
      if (k == 0) {
        for (uint32_t v = 0; v < xp_to_key_count(g, gh); ++v) {
          const uint32_t l = xp_to_key_lds(g, gh, v);
          if (lo(l, 16)) put(out + v * 16ull, &lds[l], 16);
        }
      } else {
        for (uint32_t v = 0; v < xp_to_val_count(g, gh); ++v) {
          const uint32_t l = xp_to_val_lds(g, gh, v);
          uint8_t unit[16];
          for (uint32_t j = 0; j < 16 / E; ++j)
            if (lo(l + j * rs, E)) std::memcpy(unit + j * E, &lds[l + j * rs], E);
          put(out + v * 16ull, unit, 16);
        }
      }
    }
  } else {
    const uint32_t G = xp_from_heads(g, k), rs = xp_from_row_stride(g, k);
    for (uint32_t h0 = 0; h0 < H; h0 += G) {
      const uint32_t gh = xp_min(G, H - h0);
      const uint64_t in = static_cast<uint64_t>(h0) * B * R;
      for (uint32_t v = 0; v < xp_from_load_count(g, k, gh); ++v) {
        const uint32_t l = xp_from_load_lds(g, k, v);
        if (gl(in + v * 16ull, 16) && lo(l, 16)) std::memcpy(&lds[l], src + in + v * 16ull, 16);
      }
      for (uint32_t u = 0; u < xp_from_store_count(g, gh); ++u) {
        const uint32_t l = xp_from_store_lds(g, k, gh, u), d = xp_from_store_dst(g, h0, gh, u);
        uint8_t unit[16];
        if (k == 0) {
          if (lo(l, 16)) std::memcpy(unit, &lds[l], 16);
        } else {
          for (uint32_t j = 0; j < 16 / E; ++j)
            if (lo(l + j * rs, E)) std::memcpy(unit + j * E, &lds[l + j * rs], E);
        }
        put(d, unit, 16);
      }
    }
  }
  for (uint64_t i = 0; i < piece && !bad; ++i)
    if (written[i] != 1) bad = 3;
  return bad;
}

// Head-major blocks: every unit of the piece in host order, read from and written
// to the offsets hnd_block_off gives, each access checked against the piece.
extern "C" int emu_hnd(const uint8_t* src, uint8_t* dst, int to_block, uint32_t B, uint32_t H, uint32_t R) {
  const XGeom g{B, H, R, 0, 0};
  const uint64_t piece = static_cast<uint64_t>(B) * H * R;
  std::vector<uint8_t> written(piece, 0);
  if (static_cast<uint64_t>(hnd_count(g)) * 16 != piece) return 3;
  for (uint32_t u = 0; u < hnd_count(g); ++u) {
    const uint64_t host = u * 16ull, blk = hnd_block_off(g, u);
    if (blk + 16 > piece || host + 16 > piece) return 1;
    const uint64_t so = to_block ? host : blk, d = to_block ? blk : host;
    std::memcpy(dst + d, src + so, 16);
    for (uint32_t i = 0; i < 16; ++i) written[d + i] += 1;
  }
  for (uint64_t i = 0; i < piece; ++i)
    if (written[i] != 1) return 4;
  return 0;
}
