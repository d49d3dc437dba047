// Work-list records of the dense attention launches (plain data, no HIP
// types): shared by the host runtime, the kernels and the host-side planner.
#pragma once

#include <cstdint>

// Functions shared by host code, the CPU tests and the kernels.
#if defined(__HIPCC__)
#define HC_HD __host__ __device__
#else
#define HC_HD
#endif

namespace hc {

constexpr int kMaxSrcBlocks = 32;
constexpr int kQTile = 128;    // queries per dense work unit (4 waves x 32)
constexpr int kKTile = 64;     // keys per dense KV tile

// One dense work unit: kQTile queries of one head against the contiguous key range
// [kv0, kv1) of a [keys][d] K buffer and its 8-key-grouped V buffer
// ([keys/8][d][8]).  Every unit covers at most one window block of keys, so all
// units cost about the same; a Global head's window is split into one unit per
// block and the per-block partial results are merged by the combine kernel.
// The units of a launch's last round may be cut further into pieces of whole
// key tiles (hc_plan.h).
struct DenseUnit {
  const uint16_t *k;
  const uint16_t *v;
  int32_t head;      // row block of q and o; < 0: padding unit, no work
  int32_t q0;        // first query of the unit (qn > 0: first entry of DenseArgs::qmap)
  int32_t kv0;       // first key (multiple of 8)
  int32_t kv1;       // one past the last key
  int32_t slot;      // < 0: normalise into o; else index of a partial-result slot
  int32_t out_sel;   // which of DenseArgs::o receives the unit (or its merge)
  int32_t qn;        // 0: queries q0 .. q0+kQTile-1 (clipped at L); else the qn <= kQTile
                     // tokens qmap[q0 .. q0+qn-1] (cells of the Spatial path), written
                     // directly (slot < 0)
  int32_t pad_;
};

// Partial result of one unit: unnormalised O [kQTile][d], then the running max
// (log2 units) and the row sum for each of the kQTile rows.
inline constexpr int64_t partial_floats(int d) { return (int64_t)kQTile * (d + 2); }

// Merge of the partial results of one (head, query tile).
struct CombineItem {
  int32_t head, q0;
  int32_t slot0, n_slots;  // consecutive partial slots
  int32_t out_sel, pad_;
};

}  // namespace hc
