// Layout of the Spatial path (plain C++, no HIP types): the tiling of a frame
// into work groups, the halo a work group reads in 32-key steps, and the frame
// storage of the Spatial buffers.  Shared by the host runtime and the kernels;
// compiled on its own by the CPU tests.
#pragma once

#include <algorithm>
#include <cstdint>

#include "headcast.h"

namespace hc {

// A Spatial work group covers kSpRows query rows y0 .. y0+kSpRows-1 (y0 =
// kSpRows rg) and 8 query columns x0 .. x0+7 of every frame of the block, with
// x0 = 8 c - 8 + (r & 7) for column tile c.  It reads the halo rows
// y0-r .. y0+kSpRows-1+r and 8 G key columns from column 8 gs,
// gs = c - 1 - (r >> 3): G aligned 8-key groups.
constexpr int kSpRows = 4;

inline int spatial_groups(int r) {
  const int g = (8 + 2 * r + 7) / 8;
  return g <= 1 ? 1 : (g <= 2 ? 2 : 4);
}

// Halo rows per 32-key step (a step holds whole rows of 8 G keys), halo rows
// per key frame, and steps per key frame before the ones wholly outside the
// frame are skipped.
inline int spatial_rows_per_step(int r) { return 32 / (8 * spatial_groups(r)); }
inline int spatial_halo_rows(int r) { return kSpRows + 2 * r; }
inline int spatial_steps_per_frame(int r) {
  const int rps = spatial_rows_per_step(r);
  return (spatial_halo_rows(r) + rps - 1) / rps;
}

// Steps [*s_lo, *s_hi] of the work group at y0 that hold at least one halo row
// inside the frame (the others are skipped).
inline void spatial_live_steps(int Hg, int r, int y0, int *s_lo, int *s_hi) {
  const int rps = spatial_rows_per_step(r);
  *s_lo = std::max(0, r - y0) / rps;
  *s_hi = std::min(spatial_halo_rows(r) - 1, Hg - 1 - y0 + r) / rps;
}

// Column tiles [c_lo, c_hi] of a frame of width Wg: every column lies in one.
inline void spatial_tiles(int Wg, int r, int *c_lo, int *c_hi) {
  const int o = r & 7;
  *c_lo = o == 0 ? 1 : 0;
  *c_hi = (Wg + 8 - o + 7) / 8 - 1;   // last tile with 8c-8+o < Wg
}

// Key-frame ranges a layer's Spatial launch is cut into, for `groups` work
// groups (heads x row groups x column tiles), `resident` groups the GPU holds
// at once and `frames` key frames: resident / groups ranges (at most 8) while
// the groups fill at most half of the GPU, two up to 0.55 of it, else one.
// Below half a layer's launch is one group's walk over all key frames (the
// GPU is not full); the two-range band was measured per layer at 720P and
// 1080P (0.52 and 0.53 of the GPU: 153 -> 125 us and 172 -> 156 us).
inline int spatial_split_count(int64_t groups, int64_t resident, int64_t frames) {
  if (groups <= 0 || 20 * groups > 11 * resident) return 1;
  const int64_t s = std::max<int64_t>(2, std::min<int64_t>(8, resident / groups));
  return (int)std::max<int64_t>(1, std::min<int64_t>(frames, s));
}

// Storage of a Spatial buffer: every frame is `rows` = grid_h rows of `pitch`
// = round_up(grid_w, 8) keys (row y, column x at key y pitch + x; the padding
// columns of the last 8-key group, if any, are zero), frames and heads back to
// back, with `lead` keys of zeros before the first frame and after the last.
// A work group reads halo columns outside the frame from a clamped 8-key group
// of the same row and halo rows outside the frame (at most rows_per_step - 1
// of them, in a step that also holds a row inside) from the neighbouring frame
// or the lead; all such keys are masked by index, so only the storage size
// matters.  `y0`, `x0` place the frame inside its storage (no margins).
struct SpatialGeom {
  int32_t rows, pitch, y0, x0;
  int64_t lead;
};

inline SpatialGeom spatial_geometry(const hc_config &cfg) {
  SpatialGeom g{};
  g.rows = cfg.grid_h;
  g.pitch = (cfg.grid_w + 7) / 8 * 8;
  g.y0 = 0;
  g.x0 = 0;
  const int rps = std::max(spatial_rows_per_step(cfg.spatial_radius),
                           spatial_rows_per_step(cfg.proxy_radius));
  g.lead = (int64_t)(rps - 1) * g.pitch;
  return g;
}

// The 8-key group of storage that halo column group gq (possibly outside the
// frame) is read from.
inline int spatial_clamp_group(int gq, int pitch) {
  return std::min(std::max(gq, 0), pitch / 8 - 1);
}

}  // namespace hc
