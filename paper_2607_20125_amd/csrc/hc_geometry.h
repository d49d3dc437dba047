// Layout of the Spatial path (plain C++, no HIP types): the tiling of a frame
// into work groups, the halo a work group reads, and the zero-padded frame
// storage that holds every halo.  Shared by the host runtime and the kernels;
// compiled on its own by the CPU tests.
#pragma once

#include <algorithm>
#include <cstdint>

#include "headcast.h"

namespace hc {

// A Spatial work group covers 4 query rows y0 .. y0+3 (y0 = 4 rg) and 8 query
// columns x0 .. x0+7 of every frame of the block, with x0 = 8 c - 8 + (r & 7)
// for column tile c.  It reads the halo rows y0-r .. y0+3+r and 8 G key
// columns from column 8 gs, gs = c - 1 - (r >> 3): G aligned 8-key groups.
inline int spatial_groups(int r) {
  const int g = (8 + 2 * r + 7) / 8;
  return g <= 1 ? 1 : (g <= 2 ? 2 : 4);
}

// Halo rows per 32-key tile (a tile holds whole rows of 8 G keys) and tiles
// per key frame.
inline int spatial_rows_per_tile(int r) { return 32 / (8 * spatial_groups(r)); }
inline int spatial_tiles_per_frame(int r) {
  const int rpt = spatial_rows_per_tile(r);
  return (4 + 2 * r + rpt - 1) / rpt;
}

// Column tiles [c_lo, c_hi] of a frame of width Wg: every column lies in one.
inline void spatial_tiles(int Wg, int r, int *c_lo, int *c_hi) {
  const int o = r & 7;
  *c_lo = o == 0 ? 1 : 0;
  *c_hi = (Wg + 8 - o + 7) / 8 - 1;   // last tile with 8c-8+o < Wg
}

// Padded layout of a Spatial buffer frame: row y of the frame is buffer row
// y0 + y, column x is buffer column x0 + x (x0 a multiple of 8); `rows` rows of
// `pitch` columns per frame.  The padding is zero and is never given weight;
// it lets every Spatial work group read its whole halo without clamping.
struct SpatialGeom {
  int32_t rows, pitch, y0, x0;
};

// Padding such that the halo of every Spatial work group, for the Spatial
// radius and for the proxy radius, lies inside the frame's storage: rows y0-r ..
// (its last tile's last row), column groups gs .. gs+G-1.
inline SpatialGeom spatial_geometry(const hc_config &cfg) {
  const int Hg = cfg.grid_h, Wg = cfg.grid_w, ngrp = (Wg + 7) / 8;
  int top = 0, bottom = 0, left = 0, right = 0;       // rows; 8-column groups
  for (int r : {cfg.spatial_radius, cfg.proxy_radius}) {
    const int G = spatial_groups(r);
    const int rpt = spatial_rows_per_tile(r);
    const int tpf = spatial_tiles_per_frame(r);
    const int y0_last = 4 * ((Hg + 3) / 4 - 1);
    top = std::max(top, r);
    bottom = std::max(bottom, y0_last - r + tpf * rpt - 1 - (Hg - 1));
    int c_lo, c_hi;
    spatial_tiles(Wg, r, &c_lo, &c_hi);
    left = std::max(left, -(c_lo - 1 - (r >> 3)));
    right = std::max(right, c_hi - 1 - (r >> 3) + G - 1 - (ngrp - 1));
  }
  SpatialGeom g{};
  g.rows = top + Hg + bottom;
  g.pitch = 8 * (left + ngrp + right);
  g.y0 = top;
  g.x0 = 8 * left;
  return g;
}

}  // namespace hc
