// Invariants of the Spatial path's layout (paper_2607_20125_amd/csrc/hc_geometry.h),
// on the CPU, for every grid up to 40 x 72, radius and proxy radius up to 12:
//  * the column tiles [c_lo, c_hi] cover every frame column exactly once;
//  * each work group's halo (rows y0-r .. the last row of its last 32-key tile,
//    8 G columns from 8 gs) holds the (2r+1)^2 window of each of its queries;
//  * that halo, at every row group and column tile, lies inside the padded frame
//    storage (no read outside a frame, so none outside the buffer);
//  * the padding is what the layout needs (the y0 / x0 origins are the top and
//    left margins).
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "hc_geometry.h"

using namespace hc;

static int failures = 0;
#define CHECK(cond, ...)                                   \
  do {                                                     \
    if (!(cond)) {                                         \
      std::printf("FAIL %s:%d: ", __FILE__, __LINE__);     \
      std::printf(__VA_ARGS__);                            \
      std::printf("\n");                                   \
      if (++failures > 20) std::exit(1);                   \
    }                                                      \
  } while (0)

static void check(int Hg, int Wg, int r, int rp) {
  hc_config cfg{};
  cfg.grid_h = Hg;
  cfg.grid_w = Wg;
  cfg.spatial_radius = r;
  cfg.proxy_radius = rp;
  const SpatialGeom g = spatial_geometry(cfg);
  CHECK(g.x0 % 8 == 0 && g.pitch % 8 == 0, "alignment %dx%d r=%d", Hg, Wg, r);
  CHECK(g.y0 >= 0 && g.rows >= g.y0 + Hg && g.pitch >= g.x0 + Wg, "storage %dx%d", Hg, Wg);
  for (int rr : {r, rp}) {
    const int G = spatial_groups(rr), RW = 8 * G;
    const int rpt = spatial_rows_per_tile(rr), tpf = spatial_tiles_per_frame(rr);
    CHECK(rpt * RW == 32 && tpf * rpt >= 4 + 2 * rr, "tiles r=%d", rr);
    int c_lo, c_hi;
    spatial_tiles(Wg, rr, &c_lo, &c_hi);
    std::vector<int> cover(Wg, 0);
    for (int c = c_lo; c <= c_hi; ++c) {
      const int x0 = 8 * c - 8 + (rr & 7), gs = c - 1 - (rr >> 3);
      int live = 0;
      for (int x = x0; x < x0 + 8; ++x) {
        if (x < 0 || x >= Wg) continue;
        ++cover[x];
        ++live;
        // the query's window columns lie in the halo columns
        CHECK(8 * gs <= x - rr && x + rr < 8 * gs + RW, "halo cols %dx%d r=%d c=%d x=%d", Hg, Wg,
              rr, c, x);
      }
      CHECK(live > 0, "empty column tile %dx%d r=%d c=%d", Hg, Wg, rr, c);
      // halo columns inside the storage
      CHECK(g.x0 + 8 * gs >= 0 && g.x0 + 8 * gs + RW <= g.pitch, "storage cols %dx%d r=%d c=%d",
            Hg, Wg, rr, c);
      for (int y0 = 0; y0 < Hg; y0 += 4) {
        // query rows y0..y0+3 (those inside the frame) see rows y-r..y+r
        const int h_lo = y0 - rr, h_hi = y0 - rr + tpf * rpt - 1;   // halo rows read
        for (int y = y0; y < y0 + 4 && y < Hg; ++y)
          CHECK(h_lo <= y - rr && y + rr <= h_hi, "halo rows %dx%d r=%d y=%d", Hg, Wg, rr, y);
        CHECK(g.y0 + h_lo >= 0 && g.y0 + h_hi < g.rows, "storage rows %dx%d r=%d y0=%d", Hg, Wg,
              rr, y0);
      }
    }
    for (int x = 0; x < Wg; ++x) CHECK(cover[x] == 1, "column %d covered %d times", x, cover[x]);
  }
}

int main() {
  int n = 0;
  for (int Hg = 1; Hg <= 40; ++Hg)
    for (int Wg = 1; Wg <= 72; ++Wg)
      for (int r = 0; r <= 12; r += (Hg + Wg) % 3 + 1)
        for (int rp : {0, 2, 5, 12}) {
          check(Hg, Wg, r, rp);
          ++n;
        }
  // the Wan-shaped grids
  for (int r = 0; r <= 12; ++r) {
    check(30, 52, r, 2);
    check(45, 80, r, 2);
    check(68, 120, r, 2);
    n += 3;
  }
  if (failures) return 1;
  std::printf("geometry_check: ok (%d layouts)\n", n);
  return 0;
}
