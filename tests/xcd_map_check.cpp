// Host build of the tile map in xcd_map.h: for every unit-tile count 1..64
// and row-tile count 1..40, the workgroups 0 .. rows*units-1 must reach every
// (row tile, unit tile) exactly once and never leave the grid.  Exit status 0
// on success; the first failure is printed.
#include <cstdio>
#include <vector>

#include "xcd_map.h"

int main() {
  for (int units = 1; units <= 64; ++units)
    for (int rows = 1; rows <= 40; ++rows) {
      std::vector<int> seen(rows * units, 0);
      for (int b = 0; b < rows * units; ++b) {
        const cavs::TileIdx t = cavs::xcd_tile_map(b, units);
        if (t.row_tile < 0 || t.row_tile >= rows || t.unit_tile < 0 || t.unit_tile >= units) {
          std::printf("out of range: units=%d rows=%d bid=%d -> (%d, %d)\n", units, rows, b,
                      t.row_tile, t.unit_tile);
          return 1;
        }
        if (seen[t.row_tile * units + t.unit_tile]++) {
          std::printf("repeat: units=%d rows=%d bid=%d\n", units, rows, b);
          return 1;
        }
      }
      if (units % 8 == 0)   // XCD x touches only unit tiles congruent to x mod 8
        for (int b = 0; b < rows * units; ++b)
          if (cavs::xcd_tile_map(b, units).unit_tile % 8 != b % 8) {
            std::printf("xcd order broken: units=%d bid=%d\n", units, b);
            return 1;
          }
    }
  std::printf("ok\n");
  return 0;
}
