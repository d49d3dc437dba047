// Invariants of the Spatial path's layout and tiling
// (paper_2607_20125_amd/csrc/hc_geometry.h), on the CPU, for every grid up to
// 40 x 72 and radius / proxy radius up to 12:
//  * the column tiles [c_lo, c_hi] cover every frame column exactly once, and
//    the 8 G halo columns of a tile hold the column window of each of its queries;
//  * the live steps of every row tile hold every window row (inside the frame)
//    of each of its query rows, and no step outside them does;
//  * every read stays inside the storage: rows at most rows_per_step - 1 above
//    or below the frame (covered by the buffer's leading and trailing keys,
//    frames being back to back), column groups clamped into the row;
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
  CHECK(g.pitch % 8 == 0 && g.pitch >= Wg && g.pitch < Wg + 8, "pitch %d for %d", g.pitch, Wg);
  CHECK(g.rows == Hg && g.y0 == 0 && g.x0 == 0, "frame storage %dx%d", Hg, Wg);
  for (int rr : {r, rp}) {
    const int G = spatial_groups(rr), RW = 8 * G, rps = spatial_rows_per_step(rr);
    CHECK(rps * RW == 32 && spatial_halo_rows(rr) % rps == 0, "steps r=%d", rr);
    CHECK(g.lead >= (int64_t)(rps - 1) * g.pitch, "lead %lld for r=%d", (long long)g.lead, rr);
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
        CHECK(8 * gs <= x - rr && x + rr < 8 * gs + RW, "halo cols %dx%d r=%d c=%d x=%d", Hg, Wg,
              rr, c, x);
      }
      CHECK(live > 0, "empty column tile %dx%d r=%d c=%d", Hg, Wg, rr, c);
      for (int q = gs; q < gs + G; ++q) {
        const int cq = spatial_clamp_group(q, g.pitch);
        CHECK(cq >= 0 && 8 * cq + 8 <= g.pitch, "clamped group %d of %d", cq, g.pitch);
        if (q >= 0 && 8 * q < Wg) CHECK(cq == q, "group %d inside the frame moved", q);
      }
    }
    for (int x = 0; x < Wg; ++x) CHECK(cover[x] == 1, "column %d covered %d times", x, cover[x]);
    for (int y0 = 0; y0 < Hg; y0 += kSpRows) {
      int s_lo, s_hi;
      spatial_live_steps(Hg, rr, y0, &s_lo, &s_hi);
      const int h_lo = s_lo * rps, h_hi = s_hi * rps + rps - 1;   // halo rows read
      CHECK(s_lo <= s_hi, "no live step %dx%d r=%d y0=%d", Hg, Wg, rr, y0);
      // rows read, relative to the frame
      CHECK(y0 - rr + h_lo >= -(rps - 1) && y0 - rr + h_hi <= Hg - 1 + rps - 1,
            "rows read %dx%d r=%d y0=%d: %d..%d", Hg, Wg, rr, y0, y0 - rr + h_lo, y0 - rr + h_hi);
      for (int s = 0; s < spatial_steps_per_frame(rr); ++s) {
        bool in_frame = false;
        for (int h = s * rps; h < s * rps + rps; ++h) in_frame |= y0 - rr + h >= 0 && y0 - rr + h < Hg;
        CHECK(in_frame == (s >= s_lo && s <= s_hi), "live step %d %dx%d r=%d y0=%d", s, Hg, Wg, rr, y0);
      }
      for (int y = y0; y < y0 + kSpRows && y < Hg; ++y)
        for (int yk = std::max(0, y - rr); yk <= std::min(Hg - 1, y + rr); ++yk)
          CHECK(yk - (y0 - rr) >= h_lo && yk - (y0 - rr) <= h_hi, "window row %d of %d not read", yk, y);
    }
  }
}

// The key-frame split rule: the ranges picked for the Wan-shaped grids on a
// 256-CU GPU (1024 resident groups, 21 key frames) and its bounds.
static void check_split() {
  struct Case { int64_t groups; int want; };
  // 720P: 132 groups a head (1..6 heads); 1080P: 272 (1..3); 480P: 56 (1..7)
  const Case cases[] = {{132, 7}, {264, 3}, {396, 2}, {528, 2}, {660, 1}, {792, 1},
                        {272, 3}, {544, 2}, {816, 1},
                        {56, 8}, {112, 8}, {168, 6}, {224, 4}, {280, 3}, {336, 3}, {392, 2}};
  for (const Case &k : cases)
    CHECK(spatial_split_count(k.groups, 1024, 21) == k.want, "split of %lld groups: %d, want %d",
          (long long)k.groups, spatial_split_count(k.groups, 1024, 21), k.want);
  for (int64_t g = 1; g <= 4096; ++g)
    for (int64_t fr : {1, 2, 3, 7, 21, 128}) {
      const int s = spatial_split_count(g, 1024, fr);
      CHECK(s >= 1 && s <= 8 && s <= fr, "split %d of %lld groups, %lld frames", s, (long long)g,
            (long long)fr);
      CHECK(s == 1 || g * s <= 1024 * 11 / 10 + g, "split %d overfills for %lld groups", s,
            (long long)g);
    }
  CHECK(spatial_split_count(0, 1024, 21) == 1, "no groups");
}

int main() {
  int n = 0;
  check_split();
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
