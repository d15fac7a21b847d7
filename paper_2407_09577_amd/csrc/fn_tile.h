// Workgroup -> output tile mapping of the many-row kernels (XCD-aware).
#pragma once

#include "fn_device.h"

namespace fn {

// Workgroup id -> output tile.  Consecutive workgroup ids are dispatched to the
// 8 XCDs in turn, and each XCD has its own L2.  The tile grid is cut into 8
// rectangular regions (the factorisation of 8 that keeps a region's activation
// rows plus weight columns smallest), ids are regrouped so each XCD receives one
// region, and inside a region tiles run in groups of kGroupM tile rows, so the
// tiles resident on one XCD share activation rows and weight columns in its L2.
constexpr int kXcds = 8;
constexpr int kGroupM = 4;

__device__ __forceinline__ void tile_of_block(int bid, int nblocks, int tiles_m, int tiles_n,
                                              int& tm, int& tn) {
  // Region grid rm x rn (rm * rn = 8), derived from the tile counts alone, so
  // every workgroup computes the same grid.
  int rm = 1, best = 0x7fffffff;
#pragma unroll
  for (int c = 1; c <= kXcds; c *= 2) {
    const int mm = (tiles_m + c - 1) / c, nn = (tiles_n + kXcds / c - 1) / (kXcds / c);
    if (c <= tiles_m && kXcds / c <= tiles_n && mm + nn < best) {
      best = mm + nn;
      rm = c;
    }
  }
  const int rn = kXcds / rm;
  if (best == 0x7fffffff || nblocks % kXcds != 0 || tiles_m % rm != 0 || tiles_n % rn != 0) {
    // Small or uneven grids: contiguous ranges per XCD, grouped by tile rows.
    const int q = nblocks / kXcds, r = nblocks % kXcds;
    const int x = bid % kXcds, i = bid / kXcds;
    const int logical = x * q + min(x, r) + i;
    const int per_group = kGroupM * tiles_n;
    const int group = logical / per_group;
    const int first_m = group * kGroupM;
    const int gsize = min(tiles_m - first_m, kGroupM);
    const int in_group = logical - group * per_group;
    tm = first_m + in_group % gsize;
    tn = in_group / gsize;
    return;
  }
  const int x = bid % kXcds, i = bid / kXcds;  // XCD x runs its region's tiles in order i
  const int sm = tiles_m / rm, sn = tiles_n / rn;  // region size in tiles
  const int gm = min(kGroupM, sm);
  const int per_group = gm * sn;
  const int group = i / per_group, in_group = i % per_group;
  const int first_m = group * gm;
  const int gsize = min(sm - first_m, gm);
  tm = (x / rn) * sm + first_m + in_group % gsize;
  tn = (x % rn) * sn + in_group / gsize;
}

}  // namespace fn
