// Invariants of the tail-balancing planner of the dense launches
// (paper_2607_20125_amd/csrc/hc_plan.h), on the CPU: work lists shaped like
// the runtime's (Global heads: one unit per window block and 128-query tile,
// merged per tile; Sink/Dummy heads: one unit per tile writing o; cells:
// query-mapped units) for several layer mixes and device sizes.
#include <cstdio>
#include <cstdlib>
#include <map>
#include <set>
#include <tuple>
#include <vector>

#include "hc_plan.h"

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

struct Layer {
  int L, nv, n_g, n_sd, n_cell_units;
};

// fake, disjoint head bases: addresses are only compared, never dereferenced
static const uint16_t *fake_base(int buffer, int64_t elem) {
  return reinterpret_cast<const uint16_t *>(((uintptr_t)(buffer + 1) << 40) + 2 * elem);
}

// work list as the runtime builds it before balancing (plan_dense_units with
// no CU count), plus query-mapped units shaped like cells
static void build(const Layer &ly, std::vector<DenseUnit> &units, std::vector<CombineItem> &comb) {
  const int D = 128;
  const int64_t gk = global_buffer_keys(ly.nv, ly.L), sk = sd_buffer_keys(1, ly.L);
  std::vector<HeadKV> g, sd;
  int head = 0;
  for (int i = 0; i < ly.n_g; ++i, ++head)
    g.push_back(HeadKV{head, fake_base(0, i * gk * D), fake_base(1, i * gk * D)});
  for (int i = 0; i < ly.n_sd; ++i, ++head)
    sd.push_back(HeadKV{head, fake_base(2, i * sk * D), fake_base(3, i * sk * D)});
  DensePlanShape shape;
  shape.L = ly.L;
  shape.nv = ly.nv;
  plan_dense_units(shape, g, sd, {}, 0, units, comb);
  for (int c = 0; c < ly.n_cell_units; ++c) {
    DenseUnit u{};
    u.head = head; u.q0 = c * kQTile; u.kv0 = 64 * c; u.kv1 = 64 * c + 2100; u.slot = -1;
    u.qn = 100;
    units.push_back(u);
  }
}

// what a unit computes, independent of how its keys are cut
using Key = std::tuple<int, int, int>;   // head, q0, qn
static Key key_of(const DenseUnit &u) { return Key{u.head, u.q0, u.qn}; }

static void check_layer(const Layer &ly, int n_cu, bool expect_cut) {
  std::vector<DenseUnit> units, units0;
  std::vector<CombineItem> comb, comb0;
  build(ly, units, comb);
  units0 = units;
  comb0 = comb;
  balance_units(n_cu, units, comb);
  const int n = (int)units.size();
  // 1. equal runs, one per XCD, padding only at the end of a run (the list is
  //    left as it is when the CU count is not a multiple of 8)
  if (n_cu % 8 != 0) CHECK(n == (int)units0.size(), "list changed for %d CUs", n_cu);
  else CHECK(n % 8 == 0, "list length %d not a multiple of 8", n);
  const int per = n / 8;
  for (int x = 0; x < 8 && n_cu % 8 == 0; ++x) {
    bool pad = false;
    for (int i = 0; i < per; ++i) {
      const DenseUnit &u = units[x * per + i];
      if (u.head < 0) pad = true;
      else CHECK(!pad, "work after padding in run %d", x);
    }
  }
  // 2. the key ranges of every original unit are covered exactly, in whole tiles
  std::map<std::pair<Key, int>, std::vector<std::pair<int, int>>> pieces;   // (unit, kv0 of origin)
  std::map<Key, std::vector<const DenseUnit *>> by_key;
  for (const DenseUnit &u : units)
    if (u.head >= 0) by_key[key_of(u)].push_back(&u);
  int n_cut = 0;
  for (const DenseUnit &o : units0) {
    std::vector<std::pair<int, int>> got;
    for (const DenseUnit *p : by_key[key_of(o)])
      if (p->kv0 >= o.kv0 && p->kv1 <= o.kv1) got.push_back({p->kv0, p->kv1});
    std::sort(got.begin(), got.end());
    CHECK(!got.empty(), "unit head %d q0 %d lost", o.head, o.q0);
    if (got.empty()) continue;
    CHECK(got.front().first == o.kv0 && got.back().second == o.kv1, "range not covered");
    for (size_t i = 1; i < got.size(); ++i)
      CHECK(got[i].first == got[i - 1].second, "gap or overlap in the pieces");
    for (auto &g : got) {
      CHECK((g.first - o.kv0) % kKTile == 0, "piece not at a tile boundary");
      if (got.size() > 1)
        CHECK(g.second - g.first >= 12 * kKTile || g.second == o.kv1, "piece shorter than 12 tiles");
    }
    CHECK((int)got.size() <= 8, "more than 8 pieces");
    if (got.size() > 1) {
      ++n_cut;
      CHECK(o.qn == 0, "a query-mapped unit was cut");
    }
  }
  if (expect_cut) CHECK(n_cut > 0, "no unit was cut (L %d nv %d g %d sd %d)", ly.L, ly.nv, ly.n_g, ly.n_sd);
  // 3. slots: every partial slot used once, items contiguous and small enough
  std::set<int> used;
  int max_slot = -1;
  for (const DenseUnit &u : units)
    if (u.head >= 0 && u.slot >= 0) {
      CHECK(used.insert(u.slot).second, "slot %d used twice", u.slot);
      max_slot = std::max(max_slot, u.slot);
    }
  std::vector<int> owner(max_slot + 1, -1);
  for (size_t i = 0; i < comb.size(); ++i) {
    CHECK(comb[i].n_slots >= 1 && comb[i].n_slots <= kMaxSrcBlocks, "item with %d slots", comb[i].n_slots);
    for (int s = comb[i].slot0; s < comb[i].slot0 + comb[i].n_slots; ++s) {
      CHECK(s <= max_slot && used.count(s), "item slot %d unused", s);
      if (s <= max_slot) {
        CHECK(owner[s] < 0, "slot %d in two items", s);
        owner[s] = (int)i;
      }
    }
  }
  for (int s : used) CHECK(s < (int)owner.size() && owner[s] >= 0, "slot %d in no item", s);
  // 4. each item merges exactly the pieces of its (head, query tile)
  for (const DenseUnit &u : units)
    if (u.head >= 0 && u.slot >= 0) {
      const CombineItem &it = comb[owner[u.slot]];
      CHECK(it.head == u.head && it.q0 == u.q0 && it.out_sel == u.out_sel, "piece in the wrong item");
    }
  // units that still write o directly were not cut and never had a slot
  for (const DenseUnit &u : units)
    if (u.head >= 0 && u.slot < 0) {
      bool orig = false;
      for (const DenseUnit &o : units0)
        if (key_of(o) == key_of(u) && o.kv0 == u.kv0 && o.kv1 == u.kv1 && o.slot < 0) orig = true;
      CHECK(orig, "a unit writing o is not an original one");
    }
  // 5. items of the original plan survive (Global merges)
  CHECK(comb.size() >= comb0.size(), "items lost");
  // 6. simulated end time does not grow
  auto makespan = [&](const std::vector<DenseUnit> &us) {
    const int m = (int)us.size(), slots = 2 * n_cu / 8;
    double worst = 0;
    const int p8 = m / 8, r8 = m % 8;
    for (int x = 0; x < 8; ++x) {
      const int b = x * p8 + std::min(x, r8), e = b + p8 + (x < r8 ? 1 : 0);
      std::vector<double> cost;
      for (int i = b; i < e; ++i)
        if (us[i].head >= 0) cost.push_back(plan_detail::unit_tiles(us[i]) + plan_detail::kUnitOverheadTiles);
      worst = std::max(worst, plan_detail::run_makespan(cost, slots));
    }
    return worst;
  };
  if (n_cu % 8 == 0) CHECK(makespan(units) <= makespan(units0) + 1e-9, "end time grew");
}

// ---------------------------------------------------------------------------
// Key ranges: every unit of the routed plan (Global, Sink/Dummy in one and two
// slots, cells) and of the classification sweep reads whole 64-key tiles from
// kv0; all of them must end inside the head's part of its buffer, whose keys
// per head come from the same functions the runtime allocates with.
// ---------------------------------------------------------------------------
static int n_region_plans = 0;

static void check_plan_regions(const char *what, const std::vector<DenseUnit> &units,
                               const std::vector<KeyRegion> &regions, int D, int L, int W,
                               int extra) {
  ++n_region_plans;
  const int bad = first_unit_outside(units, regions, D);
  if (bad >= 0) {
    const DenseUnit &u = units[bad];
    CHECK(false, "%s L %d W %d (%d): unit of head %d reads keys [%d, %lld) of %lld", what, L, W,
          extra, u.head, u.kv0, (long long)unit_read_end(u),
          (long long)unit_region_keys(u, regions, D));
  }
}

static void routed_regions(int L, int W, int nv, int sd_blocks, int n_cu) {
  const int D = 128, n_g = 2, n_sd = 3;
  const int64_t gk = global_buffer_keys(W, L), sk = sd_buffer_keys(sd_blocks, L);
  std::vector<HeadKV> g, sd;
  for (int i = 0; i < n_g; ++i) g.push_back(HeadKV{i, fake_base(0, i * gk * D), fake_base(1, i * gk * D)});
  for (int i = 0; i < n_sd; ++i)
    sd.push_back(HeadKV{n_g + i, fake_base(2, i * sk * D), fake_base(3, i * sk * D)});
  DensePlanShape shape;
  shape.L = L;
  shape.nv = nv;
  shape.sd_blocks = sd_blocks;
  std::vector<DenseUnit> units;
  std::vector<CombineItem> comb;
  plan_dense_units(shape, g, sd, {}, n_cu, units, comb);
  const std::vector<KeyRegion> regions = {{fake_base(0, 0), n_g, gk}, {fake_base(2, 0), n_sd, sk}};
  check_plan_regions(sd_blocks == 2 ? "routed, two Sink-Dummy slots" : "routed", units, regions,
                     D, L, W, nv);
}

static void classify_regions(int L, int W) {
  const int D = 64, H = 2;
  const int64_t tk = global_buffer_keys(W, L);
  std::vector<HeadKV> heads;
  for (int h = 0; h < H; ++h) heads.push_back(HeadKV{h, fake_base(0, h * tk * D), fake_base(1, h * tk * D)});
  std::vector<DenseUnit> units;
  std::vector<CombineItem> comb;
  plan_classify_units(L, W, heads, units, comb);
  check_plan_regions("classification", units, {{fake_base(0, 0), H, tk}}, D, L, W, 0);
}

static void cell_regions(int Hg, int Wg, int F, int W, int cs, int n_cu) {
  const int D = 128, n_sp = 2, L = F * Hg * Wg;
  const CellTables t = build_cell_tables(Hg, Wg, F, W, cs);
  std::vector<HeadKV> cells;
  for (int i = 0; i < n_sp; ++i)
    cells.push_back(HeadKV{i, fake_base(4, i * t.keys * D), fake_base(5, i * t.keys * D)});
  // the query map lists every token of the block once
  std::vector<int> seen(L, 0);
  for (int32_t tok : t.qmap) {
    CHECK(tok >= 0 && tok < L, "cell map token %d of %d", tok, L);
    if (tok >= 0 && tok < L) ++seen[tok];
  }
  for (int tok = 0; tok < L; ++tok) CHECK(seen[tok] == 1, "token %d in %d cells", tok, seen[tok]);
  for (int nv = 1; nv <= W; ++nv) {
    DensePlanShape shape;
    shape.L = L; shape.nv = nv; shape.F = F; shape.grid_h = Hg; shape.grid_w = Wg;
    shape.cell = cs; shape.cells = &t;
    std::vector<DenseUnit> units;
    std::vector<CombineItem> comb;
    plan_dense_units(shape, {}, {}, cells, n_cu, units, comb);
    check_plan_regions("cells", units, {{fake_base(4, 0), n_sp, t.keys}}, D, L, W, cs);
  }
}

// The device-side work list of hc_attention_static (closed forms of unit and
// item index) equals plan_dense_units' list before balancing, unit by unit.
static int n_static_plans = 0;

static void static_plan_matches(int L, int nv, int sd_blocks, int n_g, int n_sd) {
  ++n_static_plans;
  const int D = 64, W = 7;
  const int64_t gk = global_buffer_keys(W, L), sk = sd_buffer_keys(sd_blocks, L);
  StaticPlan p{};
  p.k_g = fake_base(0, 0); p.v_g = fake_base(1, 0); p.k_sd = fake_base(2, 0); p.v_sd = fake_base(3, 0);
  p.g_keys = gk; p.sd_keys = sk; p.d = D; p.L = L; p.nv = nv; p.nqt = (L + kQTile - 1) / kQTile;
  p.sd_parts = (sd_blocks == 2 && nv >= 2) ? 2 : 1;
  p.n_g = n_g; p.n_sd = n_sd;
  std::vector<HeadKV> g, sd;
  // heads interleaved as a table would put them: buffer slot order = head order
  int head = 0;
  for (int i = 0; i < n_g; ++i, head += 2) {
    p.g_head[i] = (int8_t)head;
    g.push_back(HeadKV{head, fake_base(0, i * gk * D), fake_base(1, i * gk * D)});
  }
  for (int i = 0; i < n_sd; ++i) {
    const int h = 2 * i + 1;
    p.sd_head[i] = (int8_t)h;
    sd.push_back(HeadKV{h, fake_base(2, i * sk * D), fake_base(3, i * sk * D)});
  }
  DensePlanShape shape;
  shape.L = L; shape.nv = nv; shape.sd_blocks = sd_blocks;
  std::vector<DenseUnit> units;
  std::vector<CombineItem> comb;
  plan_dense_units(shape, g, sd, {}, 0, units, comb);
  CHECK(static_n_units(p) == (int)units.size(), "static units %d vs %zu", static_n_units(p), units.size());
  CHECK(static_n_comb(p) == (int)comb.size(), "static items %d vs %zu", static_n_comb(p), comb.size());
  int max_slot = -1;
  for (const DenseUnit &u : units) max_slot = std::max(max_slot, u.slot);
  CHECK(static_n_slots(p) == max_slot + 1, "static slots %d vs %d", static_n_slots(p), max_slot + 1);
  for (int i = 0; i < (int)units.size() && i < static_n_units(p); ++i) {
    const DenseUnit a = static_dense_unit(p, i), &b = units[i];
    CHECK(a.k == b.k && a.v == b.v && a.head == b.head && a.q0 == b.q0 && a.kv0 == b.kv0 &&
              a.kv1 == b.kv1 && a.slot == b.slot && a.out_sel == b.out_sel && a.qn == b.qn,
          "static unit %d differs (L %d nv %d sd %d)", i, L, nv, sd_blocks);
  }
  for (int i = 0; i < (int)comb.size() && i < static_n_comb(p); ++i) {
    const CombineItem a = static_comb_item(p, i), &b = comb[i];
    CHECK(a.head == b.head && a.q0 == b.q0 && a.slot0 == b.slot0 && a.n_slots == b.n_slots &&
              a.out_sel == b.out_sel,
          "static item %d differs (L %d nv %d sd %d)", i, L, nv, sd_blocks);
  }
}

int main() {
  // the device-built work list of the no-allocation entry point
  for (int L : {8, 72, 128, 384, 4680})
    for (int nv = 1; nv <= 7; ++nv)
      for (int sdb = 1; sdb <= 2; ++sdb)
        for (auto gs : std::vector<std::pair<int, int>>{{0, 0}, {1, 0}, {0, 3}, {3, 2}, {12, 0}, {0, 12}})
          static_plan_matches(L, nv, sdb, gs.first, gs.second);
  std::printf("plan_check: %d device-built work lists match the host planner\n", n_static_plans);
  // key ranges: every L that is a multiple of 8 up to 4096, every W from 2 to 32
  for (int L = 8; L <= 4096; L += 8)
    for (int W = 2; W <= 32; ++W) {
      for (int sdb = 1; sdb <= 2; ++sdb) {
        if (sdb == 2 && W < 3) continue;   // rejected by the configuration check
        for (int nv : {1, 2, W}) routed_regions(L, W, nv, sdb, 0);
      }
      classify_regions(L, W);
    }
  // ... and after tail balancing, where units are cut into pieces
  for (int L = 8; L <= 4096; L += 8)
    for (int W : {2, 3, 7, 32})
      for (int sdb = 1; sdb <= 2; ++sdb)
        if (!(sdb == 2 && W < 3)) routed_regions(L, W, W, sdb, 256);
  // cells of 2..12 positions on grids whose blocks hold a multiple of 8 tokens
  for (int cs = 2; cs <= 12; ++cs)
    for (auto hw : std::vector<std::pair<int, int>>{{8, 8}, {5, 8}, {13, 24}, {30, 52}, {7, 3}, {1, 8}, {45, 80}})
      for (int F = 1; F <= 4; ++F) {
        if ((F * hw.first * hw.second) % 8 != 0) continue;
        for (int W : {2, 3, 7}) cell_regions(hw.first, hw.second, F, W, cs, W == 7 ? 256 : 0);
      }
  std::printf("plan_check: %d plans checked for key ranges\n", n_region_plans);

  // 480P-, 720P- and 1080P-shaped layers (L = 4680 / 10800 / 24480, W = 7)
  const std::vector<Layer> layers = {
      {4680, 7, 2, 0, 0}, {4680, 7, 1, 1, 0}, {4680, 7, 3, 4, 0}, {4680, 7, 12, 0, 0},
      {10800, 7, 2, 4, 0}, {10800, 7, 3, 5, 0}, {10800, 7, 4, 3, 0}, {10800, 7, 0, 6, 0},
      {10800, 1, 2, 4, 0}, {10800, 3, 3, 2, 0}, {24480, 7, 2, 5, 0}, {24480, 7, 3, 4, 0},
      {10800, 7, 2, 3, 37}, {128, 4, 1, 2, 0}, {40, 2, 1, 1, 0}};
  for (const Layer &ly : layers)
    for (int n_cu : {256, 304, 80, 8, 100}) {
      // layers whose last round is far from full are expected to be cut on the MI355X size
      const bool expect = n_cu == 256 && ((ly.L == 4680 && ly.n_g == 2 && ly.n_sd == 0) ||
                                          (ly.L == 4680 && ly.n_g == 1 && ly.n_sd == 1));
      check_layer(ly, n_cu, expect);
    }
  if (failures) {
    std::printf("plan_check: %d failures\n", failures);
    return 1;
  }
  std::printf("plan_check: ok\n");
  return 0;
}
