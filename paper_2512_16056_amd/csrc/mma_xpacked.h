// Index maps of the paged-KV block transforms: x-packed (key [H][R/16][B][16 bytes],
// value [H][D][B] elements; the host piece is token-major [B][H][R], R = head_dim *
// elem bytes). The dummy-task kernel stages a group of whole heads of one piece in
// a wave's LDS tile: a load phase reads 16-byte units of the group in the source's
// order into the tile, a store phase writes 16-byte units in the destination's
// order, each assembled from the tile. These functions give, for unit number u of
// a phase, the global and LDS byte offsets it touches; they are plain arithmetic,
// shared by the kernel and by a CPU test that emulates a wave over them. The
// head-major (HND) map at the end needs no tile.
#ifndef MMA_XPACKED_H_
#define MMA_XPACKED_H_

#include <stdint.h>

#if defined(__HIPCC__)
#define MMA_HD __host__ __device__
#else
#define MMA_HD
#endif

namespace mma {

struct XGeom {
  uint32_t B, H, R, E, cap;  // tokens, heads, row bytes, element bytes, LDS bytes of one wave's tile
};

MMA_HD inline uint32_t xp_min(uint32_t a, uint32_t b) { return a < b ? a : b; }
MMA_HD inline uint32_t xp_max(uint32_t a, uint32_t b) { return a > b ? a : b; }

// ---- host piece -> block. Tile: the group's token-major rows, each padded by 16 bytes.
MMA_HD inline uint32_t xp_to_heads(const XGeom& g) { return xp_max(1u, xp_min(g.H, (g.cap / g.B - 16) / g.R)); }
MMA_HD inline uint32_t xp_to_row_stride(const XGeom& g, uint32_t gh) { return gh * g.R + 16; }
// load phase: units [0, B * gh * R/16)
MMA_HD inline uint32_t xp_to_load_count(const XGeom& g, uint32_t gh) { return g.B * gh * (g.R / 16); }
MMA_HD inline void xp_to_load(const XGeom& g, uint32_t h0, uint32_t gh, uint32_t u, uint32_t* src_off,
                              uint32_t* lds_off) {
  const uint32_t ru = gh * (g.R / 16), b = u / ru, c = u - b * ru;
  *src_off = (b * g.H + h0) * g.R + c * 16;
  *lds_off = b * xp_to_row_stride(g, gh) + c * 16;
}
// store phase, key: units [0, gh * R/16 * B) of the block's group range, which
// starts at byte h0 * B * R; unit v is one 16-byte tile read
MMA_HD inline uint32_t xp_to_key_count(const XGeom& g, uint32_t gh) { return gh * (g.R / 16) * g.B; }
MMA_HD inline uint32_t xp_to_key_lds(const XGeom& g, uint32_t gh, uint32_t v) {
  const uint32_t C = g.R / 16, b = v % g.B, row = v / g.B, hl = row / C, c = row - hl * C;
  return b * xp_to_row_stride(g, gh) + hl * g.R + c * 16;
}
// store phase, value: units [0, gh * D * B*E/16); unit v gathers 16 / E elements,
// element j at lds + j * stride (stride = the tile's row stride: one token)
MMA_HD inline uint32_t xp_to_val_count(const XGeom& g, uint32_t gh) { return gh * (g.R / g.E) * (g.B * g.E / 16); }
MMA_HD inline uint32_t xp_to_val_lds(const XGeom& g, uint32_t gh, uint32_t v) {
  const uint32_t D = g.R / g.E, upr = g.B * g.E / 16, tpu = 16 / g.E;
  const uint32_t tq = v % upr, row = v / upr, hl = row / D, d = row - hl * D;
  return tq * tpu * xp_to_row_stride(g, gh) + hl * g.R + d * g.E;
}

// ---- block -> host piece. Tile: the group's block rows -- key (head, 16-byte group)
// rows of B units, value (head, dim) rows of B elements -- each padded by 16 bytes.
MMA_HD inline uint32_t xp_from_row_stride(const XGeom& g, uint32_t k) { return k == 0 ? g.B * 16 + 16 : g.B * g.E + 16; }
MMA_HD inline uint32_t xp_from_rows_per_head(const XGeom& g, uint32_t k) { return k == 0 ? g.R / 16 : g.R / g.E; }
MMA_HD inline uint32_t xp_from_heads(const XGeom& g, uint32_t k) {
  return xp_max(1u, xp_min(g.H, g.cap / (xp_from_rows_per_head(g, k) * xp_from_row_stride(g, k))));
}
// load phase: units [0, gh * rows_per_head * upr) of the block's group range
// (starting at byte h0 * B * R); unit v is read at v * 16 of that range
MMA_HD inline uint32_t xp_from_load_count(const XGeom& g, uint32_t k, uint32_t gh) {
  return gh * xp_from_rows_per_head(g, k) * (k == 0 ? g.B : g.B * g.E / 16);
}
MMA_HD inline uint32_t xp_from_load_lds(const XGeom& g, uint32_t k, uint32_t v) {
  const uint32_t upr = k == 0 ? g.B : g.B * g.E / 16, row = v / upr, q = v - row * upr;
  return row * xp_from_row_stride(g, k) + q * 16;
}
// store phase: units [0, B * gh * R/16) of the host piece's group rows
MMA_HD inline uint32_t xp_from_store_count(const XGeom& g, uint32_t gh) { return g.B * gh * (g.R / 16); }
MMA_HD inline uint32_t xp_from_store_dst(const XGeom& g, uint32_t h0, uint32_t gh, uint32_t u) {
  const uint32_t ru = gh * (g.R / 16), b = u / ru, rem = u - b * ru;
  return (b * g.H + h0) * g.R + rem * 16;
}
// key: one 16-byte tile read; value: 16 / E elements, element j at lds + j * stride
// (stride = the value tile's row stride: one dim)
MMA_HD inline uint32_t xp_from_store_lds(const XGeom& g, uint32_t k, uint32_t gh, uint32_t u) {
  const uint32_t C = g.R / 16, ru = gh * C, b = u / ru, rem = u - b * ru;
  if (k == 0) return rem * xp_from_row_stride(g, 0) + b * 16;
  const uint32_t hl = rem / C, dq = rem - hl * C, D = g.R / g.E;
  return (hl * D + dq * (16 / g.E)) * xp_from_row_stride(g, 1) + b * g.E;
}

// ---- head-major (HND) blocks: the block is [H][B][R], the host piece [B][H][R].
// Whole rows move, so there is no LDS stage: 16-byte unit u of the piece in host
// order (row u / (R/16) = t * H + h, column u % (R/16)) lives in the block at row
// h * B + t, same column.
MMA_HD inline uint32_t hnd_count(const XGeom& g) { return g.B * g.H * (g.R / 16); }
MMA_HD inline uint32_t hnd_block_off(const XGeom& g, uint32_t u) {
  const uint32_t C = g.R / 16, row = u / C, c = u - row * C, t = row / g.H, h = row - t * g.H;
  return (h * g.B + t) * g.R + c * 16;
}

}  // namespace mma

#endif  // MMA_XPACKED_H_
