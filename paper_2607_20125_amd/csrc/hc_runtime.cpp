// Host runtime of the HeadCast routed-attention library: context, validation,
// per-layer head tables and compact buffers (Sec. 4.3), work lists of the
// head-specific attention (Sec. 4.4), and the one-time online classification
// (Sec. 4.2, Eq. 2-5).  Every entry point of include/headcast.h lives here.
#include "headcast.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <functional>
#include <string>
#include <vector>

#include "hc_internal.h"
#include "hc_plan.h"

using namespace hc;

namespace {

struct DevBuf {
  void *p = nullptr;
  size_t bytes = 0;
};

struct Layer {
  bool has_types = false;
  std::vector<uint8_t> types;
  std::vector<int32_t> slot;
  std::vector<int> sd_heads, sp_heads, g_heads;
  int64_t cur_block = -1;
  DevBuf k_sd, v_sd, k_g, v_g, k_sp, v_sp;
  DevBuf units, comb;          // dense work units and combine items of the current plan
  int n_units = 0, n_comb = 0;
  int plan_nv = -1;            // valid window blocks the plan was built for
  int sp_split = 1;            // key-frame split of the Spatial work (full window)
};

struct EventPair {
  hipEvent_t a, b;
};

}  // namespace

struct hc_ctx {
  hc_config cfg{};
  int device = 0;
  float scale = 0.f;
  int L = 0, P = 0;
  SpatialGeom geo{};          // frame storage of the Spatial buffers (centred window)
  int64_t sd_keys = 0, g_keys = 0, sp_keys = 0;
  std::vector<Layer> layers;
  std::string err;
  bool profile = false;
  std::vector<EventPair> pending[HC_K_COUNT];
  std::vector<EventPair> pool;
  double prof_ms[HC_K_COUNT] = {};
  int64_t prof_n[HC_K_COUNT] = {};
  DevBuf part;                 // partial-result slots shared by all layers
  int64_t part_slots = 0;
  DevBuf sp_part, sp_ml;       // Spatial split partials shared by all layers
  int64_t sp_part_rows = 0;
  int n_cu = 0;                // compute units of the device
  // cell variant of the Spatial path (cfg.spatial_cell > 0)
  CellTables cells;
  DevBuf cell_off_d, qmap_d;   // cells.off and cells.qmap on the device
  // device memory of hc_classify_heads, allocated (and zeroed) by the first call
  // and reused by the next ones: the window in Global and in Spatial layout, the
  // four proxy outputs, the block partials, the work lists, the token statistics
  DevBuf cls_k, cls_v, cls_pk, cls_pv, cls_o[4], cls_part, cls_units, cls_comb, cls_tok;
  int cls_n_units = 0, cls_n_comb = 0;
  bool cls_done = false;       // cls_o holds the outputs of a successful classification
  void *scratch = nullptr;     // this device's fixed scratch (hc_attention_static)
};

namespace {

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

hc_status fail(hc_ctx *c, hc_status s, const char *fmt, ...) {
  if (c) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    c->err = buf;
  }
  return s;
}

#define HC_HIP(ctx, call)                                                               \
  do {                                                                                  \
    hipError_t e_ = (call);                                                             \
    if (e_ != hipSuccess)                                                               \
      return fail(ctx, e_ == hipErrorOutOfMemory ? HC_E_NOMEM : HC_E_DEVICE, "%s: %s", \
                  #call, hipGetErrorString(e_));                                        \
  } while (0)


void free_buf(DevBuf &b) {
  if (b.p) (void)hipFree(b.p);
  b = DevBuf{};
}

hc_status alloc_zero(hc_ctx *c, DevBuf &b, size_t bytes) {
  free_buf(b);
  if (bytes == 0) return HC_OK;
  hipError_t e = hipMalloc(&b.p, bytes);
  if (e != hipSuccess) {
    b.p = nullptr;
    return fail(c, HC_E_NOMEM, "hipMalloc(%zu bytes): %s", bytes, hipGetErrorString(e));
  }
  b.bytes = bytes;
  e = hipMemset(b.p, 0, bytes);
  if (e != hipSuccess) return fail(c, HC_E_DEVICE, "hipMemset: %s", hipGetErrorString(e));
  return HC_OK;
}

void free_layer(Layer &l) {
  free_buf(l.k_sd); free_buf(l.v_sd); free_buf(l.k_g); free_buf(l.v_g);
  free_buf(l.k_sp); free_buf(l.v_sp); free_buf(l.units); free_buf(l.comb);
  l.n_units = l.n_comb = 0;
  l.plan_nv = -1;
}

// --- profiling ----------------------------------------------------------------
hc_status prof_begin(hc_ctx *c, hipStream_t s, EventPair *ep) {
  if (!c->profile) return HC_OK;
  if (c->pool.empty()) {
    EventPair p;
    HC_HIP(c, hipEventCreate(&p.a));
    const hipError_t e = hipEventCreate(&p.b);
    if (e != hipSuccess) {
      (void)hipEventDestroy(p.a);
      return fail(c, HC_E_DEVICE, "hipEventCreate: %s", hipGetErrorString(e));
    }
    c->pool.push_back(p);
  }
  *ep = c->pool.back();
  c->pool.pop_back();
  HC_HIP(c, hipEventRecord(ep->a, s));
  return HC_OK;
}

hc_status prof_end(hc_ctx *c, hipStream_t s, int kind, const EventPair &ep) {
  if (!c->profile) return HC_OK;
  HC_HIP(c, hipEventRecord(ep.b, s));
  c->pending[kind].push_back(ep);
  return HC_OK;
}

template <class F>
hc_status timed_launch(hc_ctx *c, hipStream_t s, int kind, F &&launch) {
  EventPair ep{};
  hc_status st = prof_begin(c, s, &ep);
  if (st != HC_OK) return st;
  hipError_t e = launch();
  if (e != hipSuccess) return fail(c, HC_E_DEVICE, "kernel launch: %s", hipGetErrorString(e));
  return prof_end(c, s, kind, ep);
}

// --- geometry helpers ---------------------------------------------------------------
int n_valid_blocks(const hc_ctx *c, int64_t cur) {
  const int W = c->cfg.window_blocks;
  return (int)std::min<int64_t>(cur + 1, W);
}

// Block id held at logical window position i (sink first, current last).
int64_t logical_block(int64_t cur, int W, int i) {
  if (cur < W - 1) return i;
  return i == 0 ? 0 : cur - W + 1 + i;
}

hc_status check_layer(hc_ctx *c, int layer) {
  if (!c) return HC_E_INVAL;
  if (layer < 0 || layer >= c->cfg.n_layers)
    return fail(c, HC_E_INVAL, "layer %d out of range [0, %d)", layer, c->cfg.n_layers);
  return HC_OK;
}

hc_status check_types(hc_ctx *c, const uint8_t *types) {
  if (!types) return fail(c, HC_E_INVAL, "head types pointer is NULL");
  for (int h = 0; h < c->cfg.n_heads; ++h)
    if (types[h] > HC_GLOBAL) return fail(c, HC_E_INVAL, "head %d has invalid type %d", h, types[h]);
  return HC_OK;
}

int spatial_split(const hc_ctx *c, int n_sp, int radius);

// Keys of zeros before the first frame (and after the last) of a Spatial
// buffer in the centred-window layout; none in the cell-major one.
int64_t sp_lead(const hc_ctx *c) { return c->cfg.spatial_cell > 0 ? 0 : c->geo.lead; }

// First frame of a Spatial buffer (past its leading keys).
uint16_t *sp_frames(const hc_ctx *c, const DevBuf &b) {
  return b.p ? (uint16_t *)b.p + sp_lead(c) * c->cfg.head_dim : nullptr;
}

// Build the layer's head table, allocate its compact buffers and its dense work
// list (Global items first, then Sink/Dummy items: longest first).
hc_status install_types(hc_ctx *c, Layer &l, const uint8_t *types) {
  const int H = c->cfg.n_heads, D = c->cfg.head_dim;
  free_layer(l);
  l.has_types = false;
  l.types.assign(types, types + H);
  l.slot.assign(H, 0);
  l.sd_heads.clear(); l.sp_heads.clear(); l.g_heads.clear();
  for (int h = 0; h < H; ++h) {
    switch (types[h]) {
      case HC_SINK:
      case HC_DUMMY: l.slot[h] = (int)l.sd_heads.size(); l.sd_heads.push_back(h); break;
      case HC_SPATIAL: l.slot[h] = (int)l.sp_heads.size(); l.sp_heads.push_back(h); break;
      default: l.slot[h] = (int)l.g_heads.size(); l.g_heads.push_back(h); break;
    }
  }
  const size_t e2 = 2;
  hc_status st;
  if ((st = alloc_zero(c, l.k_sd, l.sd_heads.size() * c->sd_keys * D * e2)) != HC_OK) return st;
  if ((st = alloc_zero(c, l.v_sd, l.sd_heads.size() * c->sd_keys * D * e2)) != HC_OK) return st;
  if ((st = alloc_zero(c, l.k_g, l.g_heads.size() * c->g_keys * D * e2)) != HC_OK) return st;
  if ((st = alloc_zero(c, l.v_g, l.g_heads.size() * c->g_keys * D * e2)) != HC_OK) return st;
  const int64_t spk = c->cfg.spatial_cell > 0 ? c->cells.keys : c->sp_keys;
  const int64_t sp_all = l.sp_heads.empty() ? 0 : (int64_t)l.sp_heads.size() * spk + 2 * sp_lead(c);
  if ((st = alloc_zero(c, l.k_sp, sp_all * D * e2)) != HC_OK) return st;
  if ((st = alloc_zero(c, l.v_sp, sp_all * D * e2)) != HC_OK) return st;

  // Spatial work split over key frames when the layer has few Spatial heads
  l.sp_split = c->cfg.spatial_cell > 0 ? 1
                                         : spatial_split(c, (int)l.sp_heads.size(), c->cfg.spatial_radius);
  if (l.sp_split > 1) {
    const int64_t rows = (int64_t)l.sp_split * l.sp_heads.size() * c->L;
    if (rows > c->sp_part_rows) {
      HC_HIP(c, hipDeviceSynchronize());
      if ((st = alloc_zero(c, c->sp_part, (size_t)rows * D * 4)) != HC_OK) return st;
      if ((st = alloc_zero(c, c->sp_ml, (size_t)rows * 2 * 4)) != HC_OK) return st;
      c->sp_part_rows = rows;
    }
  }
  // partial slots for the largest plan of this layer (full window)
  const int64_t nqt = (c->L + kQTile - 1) / kQTile;
  const int64_t need = ((int64_t)l.g_heads.size() * c->cfg.window_blocks +
                        (int64_t)l.sd_heads.size() * (c->cfg.sd_blocks == 2 ? 2 : 0)) * nqt;
  if (need > c->part_slots) {
    HC_HIP(c, hipDeviceSynchronize());
    if ((st = alloc_zero(c, c->part, (size_t)need * partial_floats(D) * 4)) != HC_OK) return st;
    c->part_slots = need;
  }
  l.has_types = true;
  return HC_OK;
}

// Dense work of one layer with `nv` valid window blocks (hc_plan.h).
void plan_units(const hc_ctx *c, const Layer &l, int nv, std::vector<DenseUnit> &units,
                std::vector<CombineItem> &comb) {
  const int D = c->cfg.head_dim;
  auto parts = [&](const std::vector<int> &heads, const DevBuf &k, const DevBuf &v, int64_t keys) {
    std::vector<HeadKV> out;
    for (int h : heads)
      out.push_back(HeadKV{h, (const uint16_t *)k.p + (size_t)l.slot[h] * keys * D,
                           (const uint16_t *)v.p + (size_t)l.slot[h] * keys * D});
    return out;
  };
  DensePlanShape shape;
  shape.L = c->L;
  shape.nv = nv;
  shape.sd_blocks = c->cfg.sd_blocks;
  shape.F = c->cfg.frames_per_block;
  shape.grid_h = c->cfg.grid_h;
  shape.grid_w = c->cfg.grid_w;
  shape.cell = c->cfg.spatial_cell;
  shape.cells = &c->cells;
  const std::vector<HeadKV> cell_heads =
      c->cfg.spatial_cell > 0 ? parts(l.sp_heads, l.k_sp, l.v_sp, c->cells.keys)
                              : std::vector<HeadKV>{};
  plan_dense_units(shape, parts(l.g_heads, l.k_g, l.v_g, c->g_keys),
                   parts(l.sd_heads, l.k_sd, l.v_sd, c->sd_keys), cell_heads, c->n_cu, units, comb);
}

template <class T>
hc_status upload(hc_ctx *c, DevBuf &b, const std::vector<T> &v) {
  free_buf(b);
  if (v.empty()) return HC_OK;
  hc_status st = alloc_zero(c, b, v.size() * sizeof(T));
  if (st != HC_OK) return st;
  HC_HIP(c, hipMemcpy(b.p, v.data(), v.size() * sizeof(T), hipMemcpyHostToDevice));
  return HC_OK;
}

hc_status ensure_plan(hc_ctx *c, Layer &l, int nv) {
  if (l.plan_nv == nv) return HC_OK;
  std::vector<DenseUnit> units;
  std::vector<CombineItem> comb;
  plan_units(c, l, nv, units, comb);
  // every tile a unit's DMA reads (whole 64-key tiles from kv0) must lie inside
  // its head's part of the buffer
  {
    const int D = c->cfg.head_dim;
    std::vector<KeyRegion> regions = {
        {(const uint16_t *)l.k_g.p, (int64_t)l.g_heads.size(), c->g_keys},
        {(const uint16_t *)l.k_sd.p, (int64_t)l.sd_heads.size(), c->sd_keys}};
    if (c->cfg.spatial_cell > 0)
      regions.push_back({(const uint16_t *)l.k_sp.p, (int64_t)l.sp_heads.size(), c->cells.keys});
    const int bad = first_unit_outside(units, regions, D);
    if (bad >= 0) {
      const DenseUnit &u = units[bad];
      return fail(c, HC_E_STATE, "internal: work unit of head %d reads keys [%d, %lld) of %lld",
                  u.head, u.kv0, (long long)unit_read_end(u),
                  (long long)unit_region_keys(u, regions, D));
    }
  }
  if (!units.empty() || !comb.empty()) HC_HIP(c, hipDeviceSynchronize());
  // no plan until this one is complete: a failure below leaves a rebuild for
  // the next call instead of a list that does not match its counts
  l.plan_nv = -1;
  l.n_units = l.n_comb = 0;
  hc_status st;
  int64_t slots = 0;
  for (const CombineItem &it : comb) slots = std::max<int64_t>(slots, (int64_t)it.slot0 + it.n_slots);
  if (slots > c->part_slots) {
    if ((st = alloc_zero(c, c->part, (size_t)slots * partial_floats(c->cfg.head_dim) * 4)) != HC_OK)
      return st;
    c->part_slots = slots;
  }
  if ((st = upload(c, l.units, units)) != HC_OK) return st;
  if ((st = upload(c, l.comb, comb)) != HC_OK) return st;
  l.n_units = (int)units.size();
  l.n_comb = (int)comb.size();
  l.plan_nv = nv;
  return HC_OK;
}

ScatterArgs scatter_args(const hc_ctx *c, const Layer &l) {
  ScatterArgs a{};
  a.L = c->L; a.D = c->cfg.head_dim; a.Hg = c->cfg.grid_h; a.Wg = c->cfg.grid_w;
  a.geo = c->geo; a.F = c->cfg.frames_per_block;
  a.cell = c->cfg.spatial_cell; a.ncy = c->cells.ncy; a.ncx = c->cells.ncx;
  a.cell_off = (const int64_t *)c->cell_off_d.p;
  a.sd_keys = c->sd_keys; a.g_keys = c->g_keys;
  a.sp_keys = a.cell > 0 ? c->cells.keys : c->sp_keys;
  a.k_sd = (uint16_t *)l.k_sd.p; a.v_sd = (uint16_t *)l.v_sd.p;
  a.k_g = (uint16_t *)l.k_g.p; a.v_g = (uint16_t *)l.v_g.p;
  a.k_sp = sp_frames(c, l.k_sp); a.v_sp = sp_frames(c, l.v_sp);
  for (int h = 0; h < c->cfg.n_heads; ++h) {
    a.head_kind[h] = l.types[h];
    a.head_slot[h] = (uint8_t)l.slot[h];
  }
  return a;
}

// Sink-Dummy slot (L keys each) that block `b` takes in a head of archetype
// `kind` when `cur` is the current block, or -1.  One block: Sink keeps block
// 0, Dummy the current block, both in slot 0.  Two blocks: Sink keeps block 0
// in slot 0 and the current block in slot 1; Dummy keeps the previous and the
// current block in slots b mod 2.
int sd_slot(const hc_ctx *c, int kind, int64_t b, int64_t cur) {
  if (c->cfg.sd_blocks == 2) {
    if (kind == HC_SINK) return b == 0 ? 0 : (b == cur ? 1 : -1);
    return (b == cur || b == cur - 1) ? (int)(b % 2) : -1;
  }
  if (kind == HC_SINK) return b == 0 ? 0 : -1;
  return b == cur ? 0 : -1;
}

// Split a logical-order window of n = min(cur+1, W) blocks into the layer's buffers.
hc_status split_window(hc_ctx *c, Layer &l, int64_t cur, const void *k_win, const void *v_win,
                       hipStream_t s) {
  const int W = c->cfg.window_blocks;
  const int n = n_valid_blocks(c, cur);
  ScatterArgs a = scatter_args(c, l);
  a.src_k = (const uint16_t *)k_win;
  a.src_v = (const uint16_t *)v_win;
  a.n_src = n;
  for (int i = 0; i < n; ++i) {
    const int64_t b = logical_block(cur, W, i);
    a.src_slot[i] = (int8_t)hc_ring_slot(b, W);
    a.sink_slot[i] = (int8_t)sd_slot(c, HC_SINK, b, cur);
    a.dummy_slot[i] = (int8_t)sd_slot(c, HC_DUMMY, b, cur);
  }
  return timed_launch(c, s, HC_K_SCATTER, [&] { return launch_scatter(a, c->cfg.n_heads, s); });
}

// Key-frame split of a layer's Spatial work (spatial_split_count): a layer
// with few Spatial heads has fewer work groups than the GPU holds at once (four
// per CU), and the launch then takes as long as one group's walk over all W F
// key frames, so the frames are cut into ranges merged afterwards.
int spatial_split(const hc_ctx *c, int n_sp, int radius) {
  if (n_sp == 0) return 1;
  int c_lo, c_hi;
  spatial_tiles(c->cfg.grid_w, radius, &c_lo, &c_hi);
  const int64_t groups =
      (int64_t)n_sp * ((c->cfg.grid_h + kSpRows - 1) / kSpRows) * (c_hi - c_lo + 1);
  const int64_t resident = 4 * (int64_t)std::max(c->n_cu, 1);
  const int64_t frames = (int64_t)c->cfg.window_blocks * c->cfg.frames_per_block;
  return spatial_split_count(groups, resident, frames);
}

SpatialArgs spatial_args(const hc_ctx *c, int radius, int n_slots) {
  SpatialArgs a{};
  a.L = c->L; a.Hg = c->cfg.grid_h; a.Wg = c->cfg.grid_w; a.geo = c->geo;
  a.F = c->cfg.frames_per_block; a.n_slots = n_slots; a.r = radius;
  int c_hi;
  spatial_tiles(a.Wg, radius, &a.c_lo, &c_hi);
  a.n_ct = c_hi - a.c_lo + 1;
  a.n_rowgroups = (a.Hg + kSpRows - 1) / kSpRows;
  a.n_split = 1;
  a.scale_log2 = c->scale * 1.4426950408889634f;
  return a;
}

// Checks shared by hc_attention and hc_attention_static.
hc_status check_attention(hc_ctx *c, int layer, const void *q, const uint8_t *head_types,
                          const float *o) {
  hc_status st = check_layer(c, layer);
  if (st != HC_OK) return st;
  if (!q || !o) return fail(c, HC_E_INVAL, "q and o must not be NULL");
  if (!aligned16(q) || !aligned16(o)) return fail(c, HC_E_INVAL, "q and o must be 16-byte aligned");
  if ((st = check_types(c, head_types)) != HC_OK) return st;
  const Layer &l = c->layers[layer];
  if (!l.has_types) return fail(c, HC_E_STATE, "layer %d has no head table", layer);
  if (std::memcmp(head_types, l.types.data(), c->cfg.n_heads) != 0)
    return fail(c, HC_E_STATE, "head types differ from the table of layer %d", layer);
  return HC_OK;
}

// Device memory one routed layer-step works in: the dense work list and merge
// items, the partial-result slots, and the Spatial split partials.
struct LayerWork {
  const DenseUnit *units = nullptr;
  int n_units = 0;
  const CombineItem *comb = nullptr;
  int n_comb = 0;
  float *part = nullptr;
  int sp_split = 1;
  float *sp_part = nullptr, *sp_ml = nullptr;
};

// The launches of one routed layer-step (Sec. 4.4): dense units (Global,
// Sink/Dummy, cells), the merge of partials, the Spatial heads.
hc_status run_layer(hc_ctx *c, const Layer &l, int nv, const void *q, float *o,
                    const LayerWork &wk, hipStream_t s) {
  const int D = c->cfg.head_dim, H = c->cfg.n_heads;
  hc_status st;
  if (wk.n_units > 0) {
    DenseArgs a{};
    a.units = wk.units;
    a.qmap = (const int32_t *)c->qmap_d.p;
    a.q = (const uint16_t *)q;
    a.o[0] = a.o[1] = a.o[2] = o;
    a.part = wk.part;
    a.n_units = wk.n_units;
    a.L = c->L;
    a.scale_log2 = c->scale * 1.4426950408889634f;
    const DenseRole role = (int)l.g_heads.size() == H ? DenseRole::kFullWindow
                           : (c->cfg.spatial_cell > 0 || c->cfg.sd_blocks == 2)
                               ? DenseRole::kVariant
                           : (int)l.sd_heads.size() == H ? DenseRole::kSinkDummyOnly
                                                          : DenseRole::kRouted;
    st = timed_launch(c, s, HC_K_DENSE, [&] { return launch_dense(a, D, role, s); });
    if (st != HC_OK) return st;
  }
  if (wk.n_comb > 0) {
    CombineArgs a{};
    a.items = wk.comb;
    a.part = wk.part;
    a.o[0] = a.o[1] = a.o[2] = o;
    a.n_items = wk.n_comb;
    a.L = c->L;
    a.D = D;
    st = timed_launch(c, s, HC_K_COMBINE, [&] { return launch_combine(a, s); });
    if (st != HC_OK) return st;
  }
  if (!l.sp_heads.empty() && c->cfg.spatial_cell == 0) {
    SpatialArgs a = spatial_args(c, c->cfg.spatial_radius, nv);
    a.q = (const uint16_t *)q;
    a.o = o;
    a.k = sp_frames(c, l.k_sp);
    a.v = sp_frames(c, l.v_sp);
    a.head_stride = c->sp_keys * D;
    a.n_sp = (int)l.sp_heads.size();
    for (int j = 0; j < a.n_sp; ++j) a.heads[j] = (int8_t)l.sp_heads[j];
    // every split range holds at least one valid key frame
    a.n_split = std::min(wk.sp_split, nv * c->cfg.frames_per_block);
    a.part = wk.sp_part;
    a.part_ml = wk.sp_ml;
    const SpatialRole role = (int)l.sp_heads.size() == H ? SpatialRole::kSpatialOnly
                                                         : SpatialRole::kRouted;
    st = timed_launch(c, s, HC_K_SPATIAL, [&] { return launch_spatial(a, D, role, s); });
    if (st != HC_OK) return st;
  }
  return HC_OK;
}

}  // namespace

// ===========================================================================
// Public ABI
// ===========================================================================
extern "C" {

void hc_config_default(hc_config *cfg) {
  if (!cfg) return;
  hc_config d{};
  d.n_layers = 30; d.n_heads = 12; d.head_dim = 128;
  d.grid_h = 30; d.grid_w = 52; d.frames_per_block = 3; d.window_blocks = 7;
  d.spatial_radius = 4; d.proxy_radius = 2;
  d.theta_sink = d.theta_dummy = d.theta_spatial = 0.95f;
  d.theta_score = 0.755f; d.gamma = 5.0f; d.softmax_scale = 0.f;
  d.spatial_cell = 0; d.sd_blocks = 1;
  *cfg = d;
}

hc_status hc_validate_config(const hc_config *c) {
  if (!c) return HC_E_INVAL;
  if (c->n_layers < 1 || c->n_heads < 1 || c->n_heads > kMaxHeads) return HC_E_INVAL;
  if (c->head_dim != 64 && c->head_dim != 128) return HC_E_INVAL;
  if (c->grid_h < 1 || c->grid_w < 1 || c->frames_per_block < 1 || c->frames_per_block > 4)
    return HC_E_INVAL;
  if (c->window_blocks < 2 || c->window_blocks > kMaxSrcBlocks) return HC_E_INVAL;
  if (c->spatial_radius < 0 || c->spatial_radius > 12) return HC_E_INVAL;
  if (c->proxy_radius < 0 || c->proxy_radius > 12) return HC_E_INVAL;
  if (c->sd_blocks != 1 && c->sd_blocks != 2) return HC_E_INVAL;
  // The two-block Dummy set needs the previous block inside the window (block 0 plus
  // at least two recent blocks).
  if (c->sd_blocks == 2 && c->window_blocks < 3) return HC_E_INVAL;
  if (c->spatial_cell != 0) {
    if (c->spatial_cell < 2 || c->spatial_cell > 64) return HC_E_INVAL;
    if (n_cells(c->grid_h, c->spatial_cell) > 64 || n_cells(c->grid_w, c->spatial_cell) > 64)
      return HC_E_INVAL;
  }
  const int64_t L = (int64_t)c->frames_per_block * c->grid_h * c->grid_w;
  if (L % 8 != 0) return HC_E_INVAL;
  if (L * c->window_blocks + 4 * kKTile > INT32_MAX / 2) return HC_E_INVAL;
  if (!(c->softmax_scale >= 0.f) || !std::isfinite(c->softmax_scale)) return HC_E_INVAL;
  if (!std::isfinite(c->gamma) || !std::isfinite(c->theta_sink) ||
      !std::isfinite(c->theta_dummy) || !std::isfinite(c->theta_spatial) ||
      !std::isfinite(c->theta_score))
    return HC_E_INVAL;
  return HC_OK;
}

const char *hc_status_string(hc_status s) {
  switch (s) {
    case HC_OK: return "ok";
    case HC_E_INVAL: return "invalid argument";
    case HC_E_STATE: return "invalid state";
    case HC_E_ORDER: return "block out of order";
    case HC_E_NOMEM: return "out of device memory";
    case HC_E_DEVICE: return "device error";
  }
  return "unknown status";
}

const char *hc_last_error(const hc_ctx *ctx) { return ctx ? ctx->err.c_str() : ""; }

int32_t hc_ring_slot(int64_t block, int32_t W) {
  if (block < 0 || W < 2) return -1;
  if (block == 0) return 0;
  return (int32_t)(1 + (block - 1) % (W - 1));
}

hc_status hc_create(const hc_config *cfg, int device, hc_ctx **out) {
  if (!out) return HC_E_INVAL;
  *out = nullptr;
  if (hc_validate_config(cfg) != HC_OK) return HC_E_INVAL;
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || device < 0 || device >= ndev) return HC_E_DEVICE;
  if (hipSetDevice(device) != hipSuccess) return HC_E_DEVICE;
  void *scratch = nullptr;
  if (static_scratch(device, &scratch) != hipSuccess) return HC_E_DEVICE;
  hc_ctx *c = new hc_ctx;
  c->cfg = *cfg;
  c->device = device;
  c->scratch = scratch;
  c->scale = cfg->softmax_scale > 0.f ? cfg->softmax_scale : 1.0f / std::sqrt((float)cfg->head_dim);
  c->P = cfg->grid_h * cfg->grid_w;
  c->L = cfg->frames_per_block * c->P;
  c->geo = spatial_geometry(*cfg);
  // each head's part ends with a spare tile for the reads of a unit's last tile
  c->sd_keys = sd_buffer_keys(cfg->sd_blocks, c->L);
  c->g_keys = global_buffer_keys(cfg->window_blocks, c->L);
  c->sp_keys = (int64_t)cfg->window_blocks * cfg->frames_per_block * c->geo.rows * c->geo.pitch;
  if (hipDeviceGetAttribute(&c->n_cu, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess)
    c->n_cu = 0;
  c->layers.resize(cfg->n_layers);
  if (cfg->spatial_cell > 0) {
    c->cells = build_cell_tables(cfg->grid_h, cfg->grid_w, cfg->frames_per_block,
                                 cfg->window_blocks, cfg->spatial_cell);
    hc_status st = upload(c, c->cell_off_d, c->cells.off);
    if (st == HC_OK) st = upload(c, c->qmap_d, c->cells.qmap);
    if (st != HC_OK) {
      free_buf(c->cell_off_d);
      free_buf(c->qmap_d);
      delete c;
      return st;
    }
  }
  *out = c;
  return HC_OK;
}

void hc_destroy(hc_ctx *c) {
  if (!c) return;
  (void)hipSetDevice(c->device);
  (void)hipDeviceSynchronize();
  for (auto &l : c->layers) free_layer(l);
  free_buf(c->part);
  free_buf(c->sp_part);
  free_buf(c->sp_ml);
  free_buf(c->cell_off_d);
  free_buf(c->qmap_d);
  for (DevBuf *b : {&c->cls_k, &c->cls_v, &c->cls_pk, &c->cls_pv, &c->cls_o[0], &c->cls_o[1],
                    &c->cls_o[2], &c->cls_o[3], &c->cls_part, &c->cls_units, &c->cls_comb,
                    &c->cls_tok})
    free_buf(*b);
  for (int k = 0; k < HC_K_COUNT; ++k)
    for (auto &e : c->pending[k]) c->pool.push_back(e);
  for (auto &e : c->pool) {
    (void)hipEventDestroy(e.a);
    (void)hipEventDestroy(e.b);
  }
  delete c;
}

hc_status hc_set_head_types(hc_ctx *c, int layer, const uint8_t *types, int64_t cur_block,
                            const void *k_win, const void *v_win, hc_stream stream) {
  hc_status st = check_layer(c, layer);
  if (st != HC_OK) return st;
  if ((st = check_types(c, types)) != HC_OK) return st;
  if (cur_block < 0) return fail(c, HC_E_INVAL, "cur_block %lld < 0", (long long)cur_block);
  if (!k_win || !v_win) return fail(c, HC_E_INVAL, "window pointers must not be NULL");
  if (!aligned16(k_win) || !aligned16(v_win))
    return fail(c, HC_E_INVAL, "window pointers must be 16-byte aligned");
  HC_HIP(c, hipSetDevice(c->device));
  Layer &l = c->layers[layer];
  if ((st = install_types(c, l, types)) != HC_OK) {
    free_layer(l);
    l.has_types = false;
    return st;
  }
  hipStream_t s = (hipStream_t)stream;
  if ((st = split_window(c, l, cur_block, k_win, v_win, s)) != HC_OK) return st;
  l.cur_block = cur_block;
  return HC_OK;
}

hc_status hc_get_layout(const hc_ctx *cc, int layer, int32_t *head_slot, int32_t *ring) {
  hc_ctx *c = const_cast<hc_ctx *>(cc);
  hc_status st = check_layer(c, layer);
  if (st != HC_OK) return st;
  const Layer &l = c->layers[layer];
  if (!l.has_types) return fail(c, HC_E_STATE, "layer %d has no head table", layer);
  const int W = c->cfg.window_blocks;
  if (head_slot)
    for (int h = 0; h < c->cfg.n_heads; ++h) head_slot[h] = l.slot[h];
  if (ring) {
    const int n = n_valid_blocks(c, l.cur_block);
    for (int i = 0; i < W; ++i)
      ring[i] = i < n ? hc_ring_slot(logical_block(l.cur_block, W, i), W) : -1;
  }
  return HC_OK;
}

hc_status hc_append_block(hc_ctx *c, int layer, int64_t block, const void *k_blk,
                          const void *v_blk, hc_stream stream) {
  hc_status st = check_layer(c, layer);
  if (st != HC_OK) return st;
  if (!k_blk || !v_blk) return fail(c, HC_E_INVAL, "block pointers must not be NULL");
  if (!aligned16(k_blk) || !aligned16(v_blk))
    return fail(c, HC_E_INVAL, "block pointers must be 16-byte aligned");
  Layer &l = c->layers[layer];
  if (!l.has_types) return fail(c, HC_E_STATE, "layer %d has no head table", layer);
  if (block != l.cur_block && block != l.cur_block + 1)
    return fail(c, HC_E_ORDER, "block %lld after current block %lld", (long long)block,
                (long long)l.cur_block);
  HC_HIP(c, hipSetDevice(c->device));
  ScatterArgs a = scatter_args(c, l);
  a.src_k = (const uint16_t *)k_blk;
  a.src_v = (const uint16_t *)v_blk;
  a.n_src = 1;
  a.src_slot[0] = (int8_t)hc_ring_slot(block, c->cfg.window_blocks);
  a.sink_slot[0] = (int8_t)sd_slot(c, HC_SINK, block, block);
  a.dummy_slot[0] = (int8_t)sd_slot(c, HC_DUMMY, block, block);
  hipStream_t s = (hipStream_t)stream;
  st = timed_launch(c, s, HC_K_SCATTER, [&] { return launch_scatter(a, c->cfg.n_heads, s); });
  if (st != HC_OK) return st;
  l.cur_block = block;
  return HC_OK;
}

hc_status hc_attention(hc_ctx *c, int layer, const void *q, const uint8_t *head_types, float *o,
                       hc_stream stream) {
  hc_status st = check_attention(c, layer, q, head_types, o);
  if (st != HC_OK) return st;
  Layer &l = c->layers[layer];
  HC_HIP(c, hipSetDevice(c->device));
  const int nv = n_valid_blocks(c, l.cur_block);
  if ((st = ensure_plan(c, l, nv)) != HC_OK) return st;
  LayerWork wk;
  wk.units = (const DenseUnit *)l.units.p;
  wk.n_units = l.n_units;
  wk.comb = (const CombineItem *)l.comb.p;
  wk.n_comb = l.n_comb;
  wk.part = (float *)c->part.p;
  wk.sp_split = l.sp_split;
  wk.sp_part = (float *)c->sp_part.p;
  wk.sp_ml = (float *)c->sp_ml.p;
  return run_layer(c, l, nv, q, o, wk, (hipStream_t)stream);
}

hc_status hc_attention_static(hc_ctx *c, int layer, const void *q, const uint8_t *head_types,
                              float *o, hc_stream stream) {
  hc_status st = check_attention(c, layer, q, head_types, o);
  if (st != HC_OK) return st;
  if (c->cfg.spatial_cell > 0)
    return fail(c, HC_E_INVAL, "hc_attention_static: the cell variant (spatial_cell > 0) is not "
                "supported");
  Layer &l = c->layers[layer];
  const int nv = n_valid_blocks(c, l.cur_block);
  const int D = c->cfg.head_dim, F = c->cfg.frames_per_block;
  StaticPlan p{};
  p.k_g = (const uint16_t *)l.k_g.p; p.v_g = (const uint16_t *)l.v_g.p;
  p.k_sd = (const uint16_t *)l.k_sd.p; p.v_sd = (const uint16_t *)l.v_sd.p;
  p.g_keys = c->g_keys; p.sd_keys = c->sd_keys;
  p.d = D; p.L = c->L; p.nv = nv; p.nqt = (c->L + kQTile - 1) / kQTile;
  p.sd_parts = (c->cfg.sd_blocks == 2 && nv >= 2) ? 2 : 1;
  p.n_g = (int)l.g_heads.size(); p.n_sd = (int)l.sd_heads.size();
  for (int i = 0; i < p.n_g; ++i) p.g_head[i] = (int8_t)l.g_heads[i];
  for (int i = 0; i < p.n_sd; ++i) p.sd_head[i] = (int8_t)l.sd_heads[i];
  // layout of the scratch: work list, merge items, dense partials, Spatial
  // split partials and their (max, sum) pairs, each 256-byte aligned
  auto al = [](size_t b) { return (b + 255) / 256 * 256; };
  const size_t n_units = (size_t)static_n_units(p), n_comb = (size_t)static_n_comb(p);
  const size_t b_units = al(n_units * sizeof(DenseUnit)), b_comb = al(n_comb * sizeof(CombineItem));
  const size_t b_part = al((size_t)static_n_slots(p) * partial_floats(D) * sizeof(float));
  const int n_sp = (int)l.sp_heads.size();
  int split = std::min(l.sp_split, nv * F);
  auto sp_bytes = [&](int sp) {
    const size_t rows = sp > 1 ? (size_t)sp * n_sp * c->L : 0;
    return std::make_pair(al(rows * D * sizeof(float)), al(rows * 2 * sizeof(float)));
  };
  size_t need = b_units + b_comb + b_part + sp_bytes(split).first + sp_bytes(split).second;
  if (need > kStaticScratchBytes && split > 1) {
    split = 1;
    need = b_units + b_comb + b_part;
  }
  if (need > kStaticScratchBytes)
    return fail(c, HC_E_INVAL, "hc_attention_static: layer %d needs %zu bytes of scratch, the "
                "static buffer holds %zu", layer, need, (size_t)kStaticScratchBytes);
  HC_HIP(c, hipSetDevice(c->device));
  hipStream_t s = (hipStream_t)stream;
  unsigned char *base = (unsigned char *)c->scratch;
  LayerWork wk;
  wk.units = (const DenseUnit *)base;
  wk.n_units = (int)n_units;
  wk.comb = (const CombineItem *)(base + b_units);
  wk.n_comb = (int)n_comb;
  wk.part = (float *)(base + b_units + b_comb);
  wk.sp_split = split;
  wk.sp_part = (float *)(base + b_units + b_comb + b_part);
  wk.sp_ml = (float *)(base + b_units + b_comb + b_part + sp_bytes(split).first);
  HC_HIP(c, launch_static_plan(p, (DenseUnit *)wk.units, (CombineItem *)wk.comb, s));
  return run_layer(c, l, nv, q, o, wk, s);
}

namespace {

// A classification buffer of at least `bytes`, kept by the context: allocated
// and zeroed the first time, reused as is afterwards.  Padding keys of the
// window copies stay zero because later calls only rewrite real keys.
hc_status keep(hc_ctx *c, DevBuf &b, size_t bytes) {
  if (b.p && b.bytes >= bytes) return HC_OK;
  HC_HIP(c, hipDeviceSynchronize());
  return alloc_zero(c, b, bytes);
}

// Eq. 5 on one head's statistics (HC_STAT_* order, float64): the first of Sink,
// Dummy, Spatial whose test passes, else Global.
uint8_t decide_label(const hc_config &cfg, const double *st) {
  if (st[HC_STAT_COS_SINK] >= (double)cfg.theta_sink) return HC_SINK;
  if (st[HC_STAT_COS_DUMMY] >= (double)cfg.theta_dummy) return HC_DUMMY;
  if (st[HC_STAT_COS_SPATIAL] >= (double)cfg.theta_spatial &&
      st[HC_STAT_SCORE] >= (double)cfg.theta_score)
    return HC_SPATIAL;
  return HC_GLOBAL;
}

}  // namespace

hc_status hc_classify_heads(hc_ctx *c, int layer, int64_t cur_block, const void *q,
                            const void *k_win, const void *v_win, uint8_t *types_out,
                            double *stats_out, hc_stream stream) {
  hc_status st = check_layer(c, layer);
  if (st != HC_OK) return st;
  if (!q || !k_win || !v_win || !types_out)
    return fail(c, HC_E_INVAL, "q, k_win, v_win and types_out must not be NULL");
  if (!aligned16(q) || !aligned16(k_win) || !aligned16(v_win))
    return fail(c, HC_E_INVAL, "q, k_win and v_win must be 16-byte aligned");
  const int W = c->cfg.window_blocks, H = c->cfg.n_heads, D = c->cfg.head_dim, L = c->L;
  if (cur_block < W - 1)
    return fail(c, HC_E_STATE, "classification needs a full window (cur_block %lld < W-1 = %d)",
                (long long)cur_block, W - 1);
  HC_HIP(c, hipSetDevice(c->device));
  hipStream_t s = (hipStream_t)stream;
  c->cls_done = false;
  // 1. all heads in Global layout (logical order) and in Spatial layout (frames
  //    of rows of round_up(grid_w, 8) keys)
  Layer tmp;
  tmp.types.assign(H, HC_GLOBAL);
  tmp.slot.resize(H);
  for (int h = 0; h < H; ++h) tmp.slot[h] = h;
  const int64_t tkeys = global_buffer_keys(W, L);
  const size_t tbytes = (size_t)H * tkeys * D * 2;
  if ((st = keep(c, c->cls_k, tbytes)) != HC_OK || (st = keep(c, c->cls_v, tbytes)) != HC_OK)
    return st;
  void *tk = c->cls_k.p, *tv = c->cls_v.p;
  {
    ScatterArgs a = scatter_args(c, tmp);
    a.g_keys = tkeys;
    a.k_g = (uint16_t *)tk; a.v_g = (uint16_t *)tv;
    a.src_k = (const uint16_t *)k_win; a.src_v = (const uint16_t *)v_win;
    a.n_src = W;
    for (int i = 0; i < W; ++i) { a.src_slot[i] = (int8_t)i; a.sink_slot[i] = a.dummy_slot[i] = -1; }
    st = timed_launch(c, s, HC_K_SCATTER, [&] { return launch_scatter(a, H, s); });
    if (st != HC_OK) return st;
  }
  // the same window in the Spatial layout, for the Spatial proxy
  const uint16_t *sk, *sv;
  int64_t sp_stride;
  {
    const size_t pbytes = ((size_t)H * c->sp_keys + 2 * c->geo.lead) * D * 2;
    if ((st = keep(c, c->cls_pk, pbytes)) != HC_OK || (st = keep(c, c->cls_pv, pbytes)) != HC_OK)
      return st;
    // the proxy uses the centred-window layout whatever the context's variant
    uint16_t *pk = (uint16_t *)c->cls_pk.p + c->geo.lead * D;
    uint16_t *pv = (uint16_t *)c->cls_pv.p + c->geo.lead * D;
    Layer tsp = tmp;
    tsp.types.assign(H, HC_SPATIAL);
    ScatterArgs a = scatter_args(c, tsp);
    a.cell = 0;                        // the proxy uses the centred window layout
    a.sp_keys = c->sp_keys;
    a.k_sp = pk; a.v_sp = pv;
    a.src_k = (const uint16_t *)k_win; a.src_v = (const uint16_t *)v_win;
    a.n_src = W;
    for (int i = 0; i < W; ++i) { a.src_slot[i] = (int8_t)i; a.sink_slot[i] = a.dummy_slot[i] = -1; }
    st = timed_launch(c, s, HC_K_SCATTER, [&] { return launch_scatter(a, H, s); });
    if (st != HC_OK) return st;
    sk = (const uint16_t *)pk; sv = (const uint16_t *)pv;
    sp_stride = c->sp_keys * D;
  }
  // 2. O_ref, O_sink, O_dummy (Eq. 2 and the temporal proxies) in one sweep, O_spatial (r_p)
  const size_t obytes = (size_t)H * L * D * 4;
  for (int i = 0; i < 4; ++i)
    if ((st = keep(c, c->cls_o[i], obytes)) != HC_OK) return st;
  float *o_ref = (float *)c->cls_o[0].p, *o_sink = (float *)c->cls_o[1].p;
  float *o_dum = (float *)c->cls_o[2].p, *o_sp = (float *)c->cls_o[3].p;
  {
    const int nqt = (L + kQTile - 1) / kQTile;
    // One sweep: O_ref is the merge of one partial per window block; the
    // temporal proxies are the partials of block 0 (O_sink) and of the
    // current block (O_dummy) normalised on their own, so their keys are not
    // read a second time.
    std::vector<HeadKV> heads;
    for (int h = 0; h < H; ++h)
      heads.push_back(HeadKV{h, (const uint16_t *)tk + (size_t)h * tkeys * D,
                             (const uint16_t *)tv + (size_t)h * tkeys * D});
    std::vector<DenseUnit> units;
    std::vector<CombineItem> comb;
    plan_classify_units(L, W, heads, units, comb);
    {
      const std::vector<KeyRegion> regions = {{(const uint16_t *)tk, (int64_t)H, tkeys}};
      if (first_unit_outside(units, regions, D) >= 0)
        return fail(c, HC_E_STATE, "internal: a classification unit reads past its head");
    }
    if ((st = keep(c, c->cls_part, (size_t)H * nqt * W * partial_floats(D) * 4)) != HC_OK)
      return st;
    float *part = (float *)c->cls_part.p;
    // the work lists depend on the configuration only: uploaded once
    if (c->cls_n_units != (int)units.size() || c->cls_n_comb != (int)comb.size()) {
      if ((st = keep(c, c->cls_units, units.size() * sizeof(DenseUnit))) != HC_OK ||
          (st = keep(c, c->cls_comb, comb.size() * sizeof(CombineItem))) != HC_OK)
        return st;
      HC_HIP(c, hipMemcpy(c->cls_units.p, units.data(), units.size() * sizeof(DenseUnit),
                          hipMemcpyHostToDevice));
      HC_HIP(c, hipMemcpy(c->cls_comb.p, comb.data(), comb.size() * sizeof(CombineItem),
                          hipMemcpyHostToDevice));
      c->cls_n_units = (int)units.size();
      c->cls_n_comb = (int)comb.size();
    }
    void *d_units = c->cls_units.p, *d_comb = c->cls_comb.p;
    DenseArgs a{};
    a.units = (const DenseUnit *)d_units;
    a.q = (const uint16_t *)q;
    a.o[0] = o_ref; a.o[1] = o_sink; a.o[2] = o_dum;
    a.part = part;
    a.n_units = (int)units.size();
    a.L = L;
    a.scale_log2 = c->scale * 1.4426950408889634f;
    st = timed_launch(c, s, HC_K_DENSE,
                      [&] { return launch_dense(a, D, DenseRole::kClassify, s); });
    if (st != HC_OK) return st;
    CombineArgs ca{};
    ca.items = (const CombineItem *)d_comb;
    ca.part = part;
    ca.o[0] = o_ref; ca.o[1] = o_sink; ca.o[2] = o_dum;
    ca.n_items = (int)comb.size();
    ca.L = L; ca.D = D;
    st = timed_launch(c, s, HC_K_COMBINE, [&] { return launch_combine(ca, s); });
    if (st != HC_OK) return st;
  }
  {
    SpatialArgs a = spatial_args(c, c->cfg.proxy_radius, W);
    a.q = (const uint16_t *)q;
    a.o = o_sp;
    a.k = sk; a.v = sv;
    a.head_stride = sp_stride;
    a.n_sp = H;
    for (int h = 0; h < H; ++h) a.heads[h] = (int8_t)h;
    st = timed_launch(c, s, HC_K_SPATIAL,
                      [&] { return launch_spatial(a, D, SpatialRole::kClassify, s); });
    if (st != HC_OK) return st;
  }
  // 3. per-token and then per-head statistics on the device (float64), the
  // decision on the host
  if ((st = keep(c, c->cls_tok, ((size_t)H * L * 4 + (size_t)H * HC_N_STATS) * sizeof(double))) !=
      HC_OK)
    return st;
  double *tok = (double *)c->cls_tok.p;
  double *head_stats = tok + (size_t)H * L * 4;
  {
    StatsArgs a{};
    a.o_ref = o_ref; a.o_sink = o_sink; a.o_dummy = o_dum; a.o_sp = o_sp;
    a.out = tok; a.n_rows = H * L; a.D = D;
    st = timed_launch(c, s, HC_K_STATS, [&] { return launch_stats(a, s); });
    if (st != HC_OK) return st;
    ClsReduceArgs r{};
    r.tok = tok; r.out = head_stats; r.n_heads = H; r.L = L; r.D = D;
    r.gamma = (double)c->cfg.gamma;
    st = timed_launch(c, s, HC_K_STATS, [&] { return launch_cls_reduce(r, s); });
    if (st != HC_OK) return st;
  }
  static_assert(HC_N_STATS == 6 && HC_STAT_COS_SINK == 0 && HC_STAT_SCORE == 5,
                "the reduction kernel writes the statistics in HC_STAT order");
  std::vector<double> hstats((size_t)H * HC_N_STATS);
  HC_HIP(c, hipMemcpyAsync(hstats.data(), head_stats, hstats.size() * sizeof(double),
                           hipMemcpyDeviceToHost, s));
  HC_HIP(c, hipStreamSynchronize(s));
  std::vector<uint8_t> labels(H);
  for (int h = 0; h < H; ++h) labels[h] = decide_label(c->cfg, &hstats[(size_t)h * HC_N_STATS]);
  if (stats_out) std::memcpy(stats_out, hstats.data(), hstats.size() * sizeof(double));
  // 4. head table + cache split (Sec. 4.3)
  st = hc_set_head_types(c, layer, labels.data(), cur_block, k_win, v_win, stream);
  if (st != HC_OK) return st;
  std::memcpy(types_out, labels.data(), H);
  HC_HIP(c, hipStreamSynchronize(s));
  c->cls_done = true;
  return HC_OK;
}

hc_status hc_classify_outputs(hc_ctx *c, int which, float *dst, hc_stream stream) {
  if (!c) return HC_E_INVAL;
  if (which < HC_CLS_O_REF || which > HC_CLS_O_SPATIAL)
    return fail(c, HC_E_INVAL, "which = %d is not one of the four classification outputs", which);
  if (!dst || !aligned16(dst)) return fail(c, HC_E_INVAL, "dst must be a 16-byte aligned device pointer");
  if (!c->cls_done)
    return fail(c, HC_E_STATE, "no classification has completed on this context");
  const size_t bytes = (size_t)c->cfg.n_heads * c->L * c->cfg.head_dim * sizeof(float);
  HC_HIP(c, hipSetDevice(c->device));
  HC_HIP(c, hipMemcpyAsync(dst, c->cls_o[which].p, bytes, hipMemcpyDeviceToDevice,
                           (hipStream_t)stream));
  return HC_OK;
}

hc_status hc_memory_bytes(const hc_ctx *c, int64_t *bytes) {
  if (!c || !bytes) return HC_E_INVAL;
  int64_t t = 0;
  for (const auto &l : c->layers)
    t += l.k_sd.bytes + l.v_sd.bytes + l.k_g.bytes + l.v_g.bytes + l.k_sp.bytes + l.v_sp.bytes +
         l.units.bytes + l.comb.bytes;
  t += c->part.bytes + c->sp_part.bytes + c->sp_ml.bytes + c->cell_off_d.bytes + c->qmap_d.bytes;
  for (const DevBuf *b : {&c->cls_k, &c->cls_v, &c->cls_pk, &c->cls_pv, &c->cls_o[0], &c->cls_o[1],
                          &c->cls_o[2], &c->cls_o[3], &c->cls_part, &c->cls_units, &c->cls_comb,
                          &c->cls_tok})
    t += b->bytes;
  *bytes = t;
  return HC_OK;
}

hc_status hc_profile_enable(hc_ctx *c, int on) {
  if (!c) return HC_E_INVAL;
  c->profile = on != 0;
  return HC_OK;
}

hc_status hc_profile_read(hc_ctx *c, int kind, double *total_ms, int64_t *launches) {
  if (!c || kind < 0 || kind >= HC_K_COUNT || !total_ms || !launches) return HC_E_INVAL;
  HC_HIP(c, hipSetDevice(c->device));
  for (int k = 0; k < HC_K_COUNT; ++k) {
    // pairs are taken off the pending list as they are read, so a failure
    // leaves each pair in exactly one of the two lists
    auto &pend = c->pending[k];
    while (!pend.empty()) {
      const EventPair e = pend.front();
      HC_HIP(c, hipEventSynchronize(e.b));
      float ms = 0.f;
      HC_HIP(c, hipEventElapsedTime(&ms, e.a, e.b));
      c->prof_ms[k] += ms;
      c->prof_n[k] += 1;
      pend.erase(pend.begin());
      c->pool.push_back(e);
    }
  }
  *total_ms = c->prof_ms[kind];
  *launches = c->prof_n[kind];
  c->prof_ms[kind] = 0;
  c->prof_n[kind] = 0;
  return HC_OK;
}

}  // extern "C"
