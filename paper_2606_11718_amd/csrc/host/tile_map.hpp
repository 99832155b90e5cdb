// Workgroup -> output-tile map of the GEMM launch, shared by the host plan
// (test hook) and the kernel.
//
// Workgroups are dispatched to the 8 XCDs round-robin (workgroup w runs on
// XCD w mod 8). Chiplet c of G owns XCDs c*8/G .. c*8/G + 8/G - 1 and the
// output partition c (Sec. III-A: each CTA runs on the chiplet owning its
// tile). XCD x of chiplet c takes a contiguous range of that partition's
// tiles, walked in a grouped raster (group_m tile rows at a time) so that
// the tiles resident on one XCD at once share A row panels and B column
// panels in that XCD's L2.
//
// With split-K (splits > 1) every tile is computed as `splits` K ranges by
// separate workgroups of the same XCD: the XCD's range then covers tiles x
// splits virtual tiles, split-major, so that the workgroups resident
// together work on the same K range of neighbouring tiles.
#pragma once

#include <cstdint>

#if defined(__HIPCC__)
#define CCL_HD __host__ __device__ __forceinline__
#else
#define CCL_HD inline
#endif

namespace ccl {

struct TileMap {
  int32_t xcd_per_chip;   // 8 / G
  int32_t grid_c;         // Gc
  int32_t tiles_m;        // kernel tiles per partition, rows
  int32_t tiles_n;        //                              cols
  int32_t tiles_per_xcd;  // ceil(tiles_m * tiles_n * splits / xcd_per_chip)
  int32_t group_m;        // raster group height
  int32_t splits;         // K splits per tile (1: none)
};

// Returns false when workgroup wg has no tile. Otherwise pr/pc is the
// owning partition, (ti, tj) the tile inside it and split its K range.
CCL_HD bool map_tile(const TileMap& m, int64_t wg, int32_t* pr, int32_t* pc, int32_t* ti,
                     int32_t* tj, int32_t* split) {
  const int32_t xcd = (int32_t)(wg & 7);
  const int64_t slot = wg >> 3;
  const int32_t chip = xcd / m.xcd_per_chip;
  const int32_t sub = xcd - chip * m.xcd_per_chip;
  if (slot >= m.tiles_per_xcd) return false;
  const int64_t tiles = (int64_t)m.tiles_m * m.tiles_n;
  const int64_t v = (int64_t)sub * m.tiles_per_xcd + slot;
  if (v >= tiles * m.splits) return false;
  *split = (int32_t)(v / tiles);
  const int64_t t = v - (int64_t)*split * tiles;
  const int64_t per_group = (int64_t)m.group_m * m.tiles_n;
  const int32_t grp = (int32_t)(t / per_group);
  const int32_t first = grp * m.group_m;
  const int32_t gm = (m.tiles_m - first) < m.group_m ? (m.tiles_m - first) : m.group_m;
  const int32_t within = (int32_t)(t - grp * per_group);
  *ti = first + within % gm;
  *tj = within / gm;
  *pr = chip / m.grid_c;
  *pc = chip - *pr * m.grid_c;
  return true;
}

CCL_HD bool map_tile(const TileMap& m, int64_t wg, int32_t* pr, int32_t* pc, int32_t* ti,
                     int32_t* tj) {
  int32_t split;
  return map_tile(m, wg, pr, pc, ti, tj, &split);
}

}  // namespace ccl
