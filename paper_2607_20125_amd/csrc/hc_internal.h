// Internal structures shared by the host runtime (hc_runtime.cpp) and the
// gfx950 kernels (hc_dense.hip, hc_spatial.hip, hc_cache.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "headcast.h"
#include "hc_geometry.h"
#include "hc_units.h"

namespace hc {

constexpr int kMaxHeads = 64;
struct DenseArgs {
  const DenseUnit *units;
  const int32_t *qmap;     // token lists of units with qn > 0 (may be null otherwise)
  const uint16_t *q;       // [H][L][d] bf16
  float *o[3];             // [H][L][d] fp32 outputs selected by DenseUnit::out_sel
  float *part;             // partial-result slots
  int32_t n_units;
  int32_t L;
  float scale_log2;        // softmax scale * log2(e)
};

struct CombineArgs {
  const CombineItem *items;
  const float *part;
  float *o[3];
  int32_t n_items;
  int32_t L, D;
};

// Spatial path: every work group covers kSpRows query rows x one 8-column tile
// x all frames of the block for one head.  Keys come from a buffer
// K[head][slot][frame][rows][pitch][d] and V[... /8][d][8] (hc_geometry.h);
// k and v point at the first frame, geo.lead keys past the allocation's start.
struct SpatialArgs {
  const uint16_t *q;       // [H][L][d]
  float *o;                // [H][L][d]
  const uint16_t *k;       // buffer base
  const uint16_t *v;
  int64_t head_stride;     // elements between consecutive head slots (same for k and v)
  int32_t n_sp;            // heads in the buffer
  int32_t L, Hg, Wg, F;
  SpatialGeom geo;
  int32_t n_slots;         // valid window blocks
  int32_t r;               // window radius
  int32_t c_lo, n_ct;      // first column tile, number of column tiles
  int32_t n_rowgroups;     // ceil(Hg / kSpRows)
  // The key frames of the window may be split into n_split contiguous ranges,
  // one work group each; the groups then write unnormalised partial results
  // (part: [n_split][n_sp][L][d], part_ml: [n_split][n_sp][L] {max (log2), sum})
  // that spatial_merge_kernel combines into o.  n_split = 1 writes o directly.
  int32_t n_split;
  float *part;
  float *part_ml;
  float scale_log2;
  int8_t heads[kMaxHeads]; // buffer slot -> head id
};

// Scatter of source blocks into per-archetype buffers (cache split and append).
enum : uint8_t { DST_SKIP = 0, DST_SD = 1, DST_GLOBAL = 2, DST_SPATIAL = 3 };

struct ScatterArgs {
  const uint16_t *src_k;   // [H][n_src * L][d]
  const uint16_t *src_v;
  int32_t n_src;
  int32_t L, D, Hg, Wg, F;
  SpatialGeom geo;         // layout of the Spatial buffer (centred-window variant)
  // cell variant (cell > 0): the Spatial buffer is cell-major; cell (cy, cx) of
  // an ncy x ncx partition starts at key cell_off[cy * ncx + cx] and holds its
  // keys slot-major: ((slot * F + frame) * area + y_in * width + x_in)
  int32_t cell, ncy, ncx;
  const int64_t *cell_off;
  int64_t sd_keys;         // keys per head in the Sink-Dummy buffer
  int64_t g_keys;          // keys per head in the Global buffer
  int64_t sp_keys;         // keys per head in the Spatial buffer
  uint16_t *k_sd, *v_sd, *k_g, *v_g, *k_sp, *v_sp;
  int8_t src_slot[kMaxSrcBlocks];     // ring slot of each source block (Global, Spatial)
  // Sink-Dummy buffer slot (L keys each) that a source block goes to for Sink
  // and for Dummy heads, or -1 when those heads do not keep it
  int8_t sink_slot[kMaxSrcBlocks];
  int8_t dummy_slot[kMaxSrcBlocks];
  uint8_t head_kind[kMaxHeads];       // HC_SINK .. HC_GLOBAL
  uint8_t head_slot[kMaxHeads];
};

struct StatsArgs {
  const float *o_ref, *o_sink, *o_dummy, *o_sp;   // [H][L][d]
  double *out;                                     // [H][L][4]
  int32_t n_rows;                                  // H * L
  int32_t D;
};

// Per-head statistics of Eq. 3 and Eq. 4 from the per-token ones: out[h][0..5] =
// mean cos(sink, ref), mean cos(dummy, ref), mean cos(spatial, ref), the 5th
// percentile of cos(spatial, ref) (linear interpolation at rank 0.05 (L - 1)),
// MSE = sum (sp - ref)^2 / (L d), score = P5 - gamma MSE.  One work group per head.
struct ClsReduceArgs {
  const double *tok;       // [H][L][4] from the statistics kernel
  double *out;             // [H][6]
  int32_t n_heads, L, D;
  double gamma;
};

// Launchers (defined next to their kernels).  Return the launch status.
// Only separates kernel symbols (and so profiler statistics) by caller; the code is the same.
enum class DenseRole { kRouted, kFullWindow, kClassify, kVariant, kSinkDummyOnly };
hipError_t launch_dense(const DenseArgs &a, int head_dim, DenseRole role, hipStream_t s);
hipError_t launch_combine(const CombineArgs &a, hipStream_t s);
// Spatial kernel, followed by the merge of the partial results when a.n_split > 1.
// The role only separates kernel symbols by caller, as for the dense kernel.
enum class SpatialRole { kRouted, kClassify, kSpatialOnly };
hipError_t launch_spatial(const SpatialArgs &a, int head_dim, SpatialRole role, hipStream_t s);
hipError_t launch_scatter(const ScatterArgs &a, int n_heads, hipStream_t s);
hipError_t launch_stats(const StatsArgs &a, hipStream_t s);
hipError_t launch_cls_reduce(const ClsReduceArgs &a, hipStream_t s);

// The fixed device scratch of hc_attention_static (hc_static.hip).  Resolves, on
// the current device, the device address of that device's copy (once per
// device) and returns it.
constexpr size_t kStaticScratchBytes = HC_STATIC_SCRATCH_BYTES;
hipError_t static_scratch(int device, void **ptr);
// Writes the layer's dense work list and merge items (closed forms of
// hc_plan.h) into device memory.
struct StaticPlan;
hipError_t launch_static_plan(const StaticPlan &p, DenseUnit *units, CombineItem *comb,
                              hipStream_t s);

}  // namespace hc
