// Host-side planning of the dense launches (plain C++, no HIP): the keys per
// head of the buffers the dense kernel reads (Sec. 4.3 buffers), the cell
// tables of the cell variant, the work lists of the routed step (Sec. 4.4) and
// of the classification sweep (Sec. 4.2), the check that every unit stays
// inside its head's part of a buffer, and the tail balancing of the unit runs
// the 8 XCDs execute.  Used by the runtime; compiled on its own by the CPU tests.
#pragma once

#include <algorithm>
#include <cstdint>
#include <functional>
#include <vector>

#include "hc_units.h"

namespace hc {

inline int64_t round_up_tiles(int64_t keys) { return (keys + kKTile - 1) / kKTile * kKTile; }

// ---------------------------------------------------------------------------
// Keys per head of the buffers the dense kernel reads.  A unit's DMA moves
// whole kKTile-key tiles from kv0, so it reads up to kKTile - 1 keys past kv1:
// with two Sink-Dummy slots the second slot's unit starts at key L and its
// tiles end as late as L + round_up(L) > round_up(2 L) whenever L is not a
// multiple of kKTile.  Every buffer therefore ends each head with one spare tile.
// ---------------------------------------------------------------------------
inline int64_t sd_buffer_keys(int sd_blocks, int64_t L) {
  return round_up_tiles((int64_t)sd_blocks * L) + kKTile;
}
inline int64_t global_buffer_keys(int n_blocks, int64_t L) {
  return round_up_tiles((int64_t)n_blocks * L) + kKTile;
}

// ---------------------------------------------------------------------------
// Cell variant of the Spatial path: round(N / c) cells per axis (halves
// rounded up, at least one); all cells are c wide except the last, which ends
// at N.  A cell's keys are stored slot-major and padded to whole tiles; the
// query map lists the block's tokens cell by cell (frame-major inside a cell).
// ---------------------------------------------------------------------------
inline int n_cells(int N, int c) { return std::max(1, (2 * N + c) / (2 * c)); }

struct CellTables {
  int ncy = 0, ncx = 0;              // cells per column / per row
  std::vector<int64_t> off;          // first key of each cell (row-major cells)
  std::vector<int32_t> q0;           // first entry of each cell in qmap
  std::vector<int32_t> qmap;         // tokens cell by cell
  int64_t keys = 0;                  // keys per head of the cell-major buffer
  int cell_h(int cy, int Hg, int cs) const { return cy == ncy - 1 ? Hg - cy * cs : cs; }
  int cell_w(int cx, int Wg, int cs) const { return cx == ncx - 1 ? Wg - cx * cs : cs; }
};

inline CellTables build_cell_tables(int Hg, int Wg, int F, int W, int cs) {
  CellTables t;
  t.ncy = n_cells(Hg, cs);
  t.ncx = n_cells(Wg, cs);
  int64_t off = 0;
  for (int cy = 0; cy < t.ncy; ++cy)
    for (int cx = 0; cx < t.ncx; ++cx) {
      const int y0 = cy * cs, y1 = y0 + t.cell_h(cy, Hg, cs);
      const int x0 = cx * cs, x1 = x0 + t.cell_w(cx, Wg, cs);
      t.off.push_back(off);
      off += round_up_tiles((int64_t)W * F * (y1 - y0) * (x1 - x0));
      t.q0.push_back((int32_t)t.qmap.size());
      for (int f = 0; f < F; ++f)
        for (int y = y0; y < y1; ++y)
          for (int x = x0; x < x1; ++x) t.qmap.push_back(f * Hg * Wg + y * Wg + x);
    }
  t.keys = off + kKTile;   // the spare tile, as in the other buffers
  return t;
}

// ---------------------------------------------------------------------------
// Work lists.  A head's part of a buffer is given by its K and V bases.
// ---------------------------------------------------------------------------
struct HeadKV {
  int head;
  const uint16_t *k, *v;
};

struct DensePlanShape {
  int L = 0;                 // tokens per block
  int nv = 0;                // valid window blocks
  int sd_blocks = 1;         // Sink-Dummy slots per head (1 or 2)
  int F = 1, grid_h = 0, grid_w = 0, cell = 0;   // cell variant (cell > 0)
  const CellTables *cells = nullptr;
};

// Dense work of one routed layer: Global heads get one unit per window block
// and 128-query tile (partials merged per tile), Sink/Dummy heads one unit per
// tile over their block (per block slot in the two-block variant once a second
// block exists, merged like a Global head), cells one query-mapped unit per
// 128 queries of a cell.  Units are ordered (head, key block, query tile) so
// that neighbouring units read the same K/V.  Then tail-balanced for n_cu CUs.
inline void balance_units(int n_cu, std::vector<DenseUnit> &units, std::vector<CombineItem> &comb);

inline void plan_dense_units(const DensePlanShape &s, const std::vector<HeadKV> &global,
                             const std::vector<HeadKV> &sink_dummy,
                             const std::vector<HeadKV> &cell_heads, int n_cu,
                             std::vector<DenseUnit> &units, std::vector<CombineItem> &comb) {
  const int L = s.L, nv = s.nv;
  const int nqt = (L + kQTile - 1) / kQTile;
  units.clear();
  comb.clear();
  int slot = 0;
  for (const HeadKV &h : global) {
    for (int blk = 0; blk < nv; ++blk)
      for (int qt = 0; qt < nqt; ++qt) {
        DenseUnit u{};
        u.k = h.k; u.v = h.v; u.head = h.head; u.q0 = qt * kQTile;
        u.kv0 = blk * L; u.kv1 = (blk + 1) * L;
        u.slot = nv > 1 ? slot + qt * nv + blk : -1;
        units.push_back(u);
      }
    if (nv > 1) {
      for (int qt = 0; qt < nqt; ++qt)
        comb.push_back(CombineItem{h.head, qt * kQTile, slot + qt * nv, nv, 0, 0});
      slot += nqt * nv;
    }
  }
  const int sd_parts = (s.sd_blocks == 2 && nv >= 2) ? 2 : 1;
  for (const HeadKV &h : sink_dummy) {
    for (int part = 0; part < sd_parts; ++part)
      for (int qt = 0; qt < nqt; ++qt) {
        DenseUnit u{};
        u.k = h.k; u.v = h.v; u.head = h.head; u.q0 = qt * kQTile;
        u.kv0 = part * L; u.kv1 = (part + 1) * L;
        u.slot = sd_parts > 1 ? slot + qt * sd_parts + part : -1;
        units.push_back(u);
      }
    if (sd_parts > 1) {
      for (int qt = 0; qt < nqt; ++qt)
        comb.push_back(CombineItem{h.head, qt * kQTile, slot + qt * sd_parts, sd_parts, 0, 0});
      slot += nqt * sd_parts;
    }
  }
  if (s.cell > 0 && s.cells) {
    const CellTables &t = *s.cells;
    for (const HeadKV &h : cell_heads)
      for (int cy = 0; cy < t.ncy; ++cy)
        for (int cx = 0; cx < t.ncx; ++cx) {
          const int id = cy * t.ncx + cx;
          const int area = t.cell_h(cy, s.grid_h, s.cell) * t.cell_w(cx, s.grid_w, s.cell);
          const int nq = s.F * area;
          for (int q = 0; q < nq; q += kQTile) {
            DenseUnit u{};
            u.k = h.k; u.v = h.v; u.head = h.head; u.q0 = t.q0[id] + q;
            u.kv0 = (int32_t)t.off[id];
            u.kv1 = u.kv0 + nv * s.F * area;
            u.slot = -1;
            u.qn = std::min(kQTile, nq - q);
            units.push_back(u);
          }
        }
  }
  balance_units(n_cu, units, comb);
}

// ---------------------------------------------------------------------------
// The same routed work list (before tail balancing) as a closed form of the
// unit index, for plans built on the device (hc_attention_static): unit i and
// merge item i of a layer from the head lists and buffer bases alone.  The
// order is plan_dense_units' (Global heads, then Sink/Dummy heads).
// ---------------------------------------------------------------------------
struct StaticPlan {
  const uint16_t *k_g, *v_g, *k_sd, *v_sd;   // buffer bases; head slot s at s * keys * d
  int64_t g_keys, sd_keys;
  int32_t d, L, nv, nqt, sd_parts, n_g, n_sd;
  int8_t g_head[64], sd_head[64];            // head id of each buffer slot
};

inline HC_HD int static_n_units(const StaticPlan &p) {
  return (p.n_g * p.nv + p.n_sd * p.sd_parts) * p.nqt;
}
inline HC_HD int static_n_comb(const StaticPlan &p) {
  return ((p.nv > 1 ? p.n_g : 0) + (p.sd_parts > 1 ? p.n_sd : 0)) * p.nqt;
}
inline HC_HD int static_n_slots(const StaticPlan &p) {
  return ((p.nv > 1 ? p.n_g * p.nv : 0) + (p.sd_parts > 1 ? p.n_sd * p.sd_parts : 0)) * p.nqt;
}

inline HC_HD DenseUnit static_dense_unit(const StaticPlan &p, int i) {
  DenseUnit u{};
  const int ng_units = p.n_g * p.nv * p.nqt;
  const int g_slots = p.nv > 1 ? ng_units : 0;
  if (i < ng_units) {                         // Global: (head, block, query tile)
    const int qt = i % p.nqt, blk = (i / p.nqt) % p.nv, gi = i / (p.nqt * p.nv);
    u.k = p.k_g + (int64_t)gi * p.g_keys * p.d;
    u.v = p.v_g + (int64_t)gi * p.g_keys * p.d;
    u.head = p.g_head[gi];
    u.kv0 = blk * p.L;
    u.slot = p.nv > 1 ? gi * p.nqt * p.nv + qt * p.nv + blk : -1;
    u.q0 = qt * kQTile;
  } else {                                    // Sink/Dummy: (head, block slot, query tile)
    const int j = i - ng_units;
    const int qt = j % p.nqt, part = (j / p.nqt) % p.sd_parts, si = j / (p.nqt * p.sd_parts);
    u.k = p.k_sd + (int64_t)si * p.sd_keys * p.d;
    u.v = p.v_sd + (int64_t)si * p.sd_keys * p.d;
    u.head = p.sd_head[si];
    u.kv0 = part * p.L;
    u.slot = p.sd_parts > 1 ? g_slots + si * p.nqt * p.sd_parts + qt * p.sd_parts + part : -1;
    u.q0 = qt * kQTile;
  }
  u.kv1 = u.kv0 + p.L;
  return u;
}

inline HC_HD CombineItem static_comb_item(const StaticPlan &p, int i) {
  const int ng_items = p.nv > 1 ? p.n_g * p.nqt : 0;
  const int g_slots = p.nv > 1 ? p.n_g * p.nv * p.nqt : 0;
  CombineItem it{};
  if (i < ng_items) {
    const int qt = i % p.nqt, gi = i / p.nqt;
    it.head = p.g_head[gi];
    it.q0 = qt * kQTile;
    it.slot0 = gi * p.nqt * p.nv + qt * p.nv;
    it.n_slots = p.nv;
  } else {
    const int j = i - ng_items;
    const int qt = j % p.nqt, si = j / p.nqt;
    it.head = p.sd_head[si];
    it.q0 = qt * kQTile;
    it.slot0 = g_slots + si * p.nqt * p.sd_parts + qt * p.sd_parts;
    it.n_slots = p.sd_parts;
  }
  return it;
}

// The classification sweep (Sec. 4.2): per head one unit per window block and
// query tile over the window in Global layout; O_ref is the merge of all W
// partials of a tile (output 0), O_sink the block-0 partial (output 1) and
// O_dummy the current-block partial (output 2), each normalised on its own.
inline void plan_classify_units(int L, int W, const std::vector<HeadKV> &heads,
                                std::vector<DenseUnit> &units, std::vector<CombineItem> &comb) {
  const int nqt = (L + kQTile - 1) / kQTile;
  units.clear();
  comb.clear();
  for (int hi = 0; hi < (int)heads.size(); ++hi) {
    const HeadKV &h = heads[hi];
    for (int blk = 0; blk < W; ++blk)
      for (int qt = 0; qt < nqt; ++qt) {
        DenseUnit u{};
        u.k = h.k; u.v = h.v; u.head = h.head; u.q0 = qt * kQTile;
        u.kv0 = blk * L; u.kv1 = (blk + 1) * L;
        u.slot = (hi * nqt + qt) * W + blk;
        units.push_back(u);
      }
    for (int qt = 0; qt < nqt; ++qt) {
      const int s0 = (hi * nqt + qt) * W;
      comb.push_back(CombineItem{h.head, qt * kQTile, s0, W, 0, 0});
      comb.push_back(CombineItem{h.head, qt * kQTile, s0, 1, 1, 0});
      comb.push_back(CombineItem{h.head, qt * kQTile, s0 + W - 1, 1, 2, 0});
    }
  }
}

// ---------------------------------------------------------------------------
// Every tile a unit's DMA reads (whole kKTile-key tiles from kv0) must lie
// inside its head's part of a buffer.  A buffer is n_heads parts of `keys`
// keys of d elements from `base`; a unit's k must be the base of one part.
// Addresses are compared as integers (no buffer is dereferenced).
// ---------------------------------------------------------------------------
struct KeyRegion {
  const uint16_t *base;
  int64_t n_heads, keys;
};

// keys of the part u.k starts, or -1 when u.k is no part's base
inline int64_t unit_region_keys(const DenseUnit &u, const std::vector<KeyRegion> &regions, int d) {
  const uintptr_t k = reinterpret_cast<uintptr_t>(u.k);
  for (const KeyRegion &r : regions) {
    const uintptr_t b = reinterpret_cast<uintptr_t>(r.base);
    const uintptr_t part = (uintptr_t)r.keys * d * sizeof(uint16_t);
    if (!r.base || part == 0 || k < b || k >= b + part * r.n_heads) continue;
    if ((k - b) % part == 0) return r.keys;
  }
  return -1;
}

// one past the last key a unit's DMA reads
inline int64_t unit_read_end(const DenseUnit &u) {
  return u.kv0 + round_up_tiles((int64_t)u.kv1 - u.kv0);
}

// index of the first unit (padding units aside) that reads outside its head's
// part, or -1 when all stay inside
inline int first_unit_outside(const std::vector<DenseUnit> &units,
                              const std::vector<KeyRegion> &regions, int d) {
  for (size_t i = 0; i < units.size(); ++i) {
    const DenseUnit &u = units[i];
    if (u.head < 0) continue;
    const int64_t keys = unit_region_keys(u, regions, d);
    if (keys < 0 || u.kv0 < 0 || u.kv1 < u.kv0 || unit_read_end(u) > keys) return (int)i;
  }
  return -1;
}

// ---------------------------------------------------------------------------
// Tail balancing of a dense launch.  Work groups are dealt round-robin to the
// 8 XCDs and the kernel maps them so that XCD x runs a contiguous run of the
// unit list in order, `per_xcd` (two per CU) at a time.  With equal units the
// last round of a run is partly empty.  For each run, the tail (its last
// partial round, or that plus one full round) is cut into pieces of whole key
// tiles when a list-scheduling simulation says the run then ends earlier; each
// piece writes a partial slot and the pieces are merged by the combine kernel
// like the per-block partials of a Global head.  Runs are padded with no-op
// units (head < 0) to one length so the mapping stays run x -> XCD x.
// ---------------------------------------------------------------------------
namespace plan_detail {

constexpr double kUnitOverheadTiles = 4.0;   // fixed cost of a unit (Q load, fill, store)
constexpr int kMinPieceTiles = 12;
constexpr int kMaxPieces = 8;

inline int unit_tiles(const DenseUnit &u) { return (u.kv1 - u.kv0 + kKTile - 1) / kKTile; }

inline double run_makespan(const std::vector<double> &cost, int slots) {
  std::vector<double> heap(slots, 0.0);   // min-heap of slot free times
  std::make_heap(heap.begin(), heap.end(), std::greater<double>());
  double end = 0.0;
  for (double w : cost) {
    std::pop_heap(heap.begin(), heap.end(), std::greater<double>());
    heap.back() += w;
    end = std::max(end, heap.back());
    std::push_heap(heap.begin(), heap.end(), std::greater<double>());
  }
  return end;
}

}  // namespace plan_detail

// n_cu: compute units of the device (a multiple of 8; otherwise the list is left as is).
inline void balance_units(int n_cu, std::vector<DenseUnit> &units, std::vector<CombineItem> &comb) {
  using namespace plan_detail;
  const int n = (int)units.size();
  if (n_cu <= 0 || n_cu % 8 != 0 || n == 0) return;
  const int slots = 2 * n_cu / 8;
  // item of every unit: the combine item holding its slot, or -1 (writes o)
  std::vector<int> item(n, -1);
  {
    std::vector<int> of_slot;
    for (int i = 0; i < (int)comb.size(); ++i)
      for (int j = 0; j < comb[i].n_slots; ++j) {
        const int sl = comb[i].slot0 + j;
        if (sl >= (int)of_slot.size()) of_slot.resize(sl + 1, -1);
        of_slot[sl] = i;
      }
    for (int i = 0; i < n; ++i)
      if (units[i].slot >= 0) item[i] = of_slot[units[i].slot];
  }
  std::vector<int> item_n(comb.size());
  for (size_t i = 0; i < comb.size(); ++i) item_n[i] = comb[i].n_slots;

  struct Piece { DenseUnit u; int item; };
  std::vector<std::vector<Piece>> runs(8);
  const int per = n / 8, rem = n % 8;
  size_t longest = 0;
  for (int x = 0; x < 8; ++x) {
    const int b = x * per + std::min(x, rem), e = b + per + (x < rem ? 1 : 0);
    std::vector<double> base;
    for (int i = b; i < e; ++i) base.push_back(unit_tiles(units[i]) + kUnitOverheadTiles);
    const int m = e - b;
    // best (suffix length j, pieces k) by simulated end time
    double best = run_makespan(base, slots);
    int best_j = 0, best_k = 1;
    const int tail = m % slots;
    for (int j : {tail, tail + slots}) {
      if (j <= 0 || j > m) continue;
      for (int k = 2; k <= kMaxPieces; ++k) {
        std::vector<double> cost(base.begin(), base.end() - j);
        for (int i = e - j; i < e; ++i) {
          const int nt = unit_tiles(units[i]);
          const bool can = units[i].qn == 0 && nt >= k * kMinPieceTiles;
          const int kk = can ? k : 1;
          for (int p = 0; p < kk; ++p)
            cost.push_back((nt * (p + 1) / kk - nt * p / kk) + kUnitOverheadTiles);
        }
        const double t = run_makespan(cost, slots);
        if (t < best * 0.99) { best = t; best_j = j; best_k = k; }
      }
    }
    std::vector<Piece> &r = runs[x];
    for (int i = b; i < e; ++i) {
      const DenseUnit &u = units[i];
      const int nt = unit_tiles(u);
      int k = (i >= e - best_j && u.qn == 0 && nt >= best_k * kMinPieceTiles) ? best_k : 1;
      if (k > 1 && item[i] >= 0 && item_n[item[i]] + k - 1 > kMaxSrcBlocks) k = 1;
      if (k == 1) { r.push_back({u, item[i]}); continue; }
      int it = item[i];
      if (it < 0) {               // a unit writing o directly gets an item of its own
        it = (int)comb.size();
        comb.push_back(CombineItem{u.head, u.q0, 0, 0, u.out_sel, 0});
        item_n.push_back(1);
      }
      item_n[it] += k - 1;
      for (int p = 0; p < k; ++p) {
        DenseUnit q = u;
        q.kv0 = u.kv0 + kKTile * (nt * p / k);
        q.kv1 = std::min(u.kv1, u.kv0 + kKTile * (nt * (p + 1) / k));
        r.push_back({q, it});
      }
    }
    longest = std::max(longest, r.size());
  }
  // slots: consecutive per item
  std::vector<int> next(comb.size());
  int slot = 0;
  for (size_t i = 0; i < comb.size(); ++i) {
    comb[i].slot0 = slot;
    comb[i].n_slots = item_n[i];
    next[i] = slot;
    slot += item_n[i];
  }
  units.clear();
  for (int x = 0; x < 8; ++x) {
    for (Piece &p : runs[x]) {
      p.u.slot = p.item >= 0 ? next[p.item]++ : -1;
      units.push_back(p.u);
    }
    DenseUnit none{};
    none.head = -1;
    for (size_t i = runs[x].size(); i < longest; ++i) units.push_back(none);
  }
}

}  // namespace hc
