// Host-side planning of a dense launch's work list (plain C++, no HIP): the
// tail balancing of the unit runs the 8 XCDs execute.  Used by the runtime;
// compiled on its own by the CPU tests.
#pragma once

#include <algorithm>
#include <functional>
#include <vector>

#include "hc_units.h"

namespace hc {

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
