// Workgroup -> (row tile, unit tile) map of the tiled level and lazy
// products.  Plain integer code: constexpr functions compile for the GPU and
// for the host alike, so the map is checked on the CPU for every tile count
// (tests/xcd_map_check.cpp).
//
// Workgroup b of a launch runs on XCD b % 8 (round-robin dispatch), and each
// XCD has its own L2.  Tiles are mapped so that XCD x only touches unit tiles
// x, x+8, ...: each L2 then holds 1/8 of the weight columns instead of all.
// With a unit-tile count that is not a multiple of 8 (narrow layers) the
// plain row-major order is used: the mapping above needs at least 8 unit
// tiles and would otherwise divide by zero.  For a grid of exactly
// n_row_tiles * n_unit_tiles workgroups the map is a bijection.
#pragma once

namespace cavs {

struct TileIdx {
  int row_tile, unit_tile;
};

constexpr TileIdx xcd_tile_map(int bid, int n_unit_tiles) {
  if (n_unit_tiles & 7) return TileIdx{bid / n_unit_tiles, bid % n_unit_tiles};
  const int xcd = bid & 7, local = bid >> 3, per = n_unit_tiles >> 3;
  return TileIdx{local / per, xcd + 8 * (local % per)};
}

}  // namespace cavs
