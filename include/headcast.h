/*
 * headcast.h -- C ABI of the HeadCast routed-attention library for MI355X (gfx950).
 *
 * HeadCast (arXiv 2607.20125) classifies every attention head of an
 * autoregressive video-diffusion model once (Sec. 4.2), splits the KV cache
 * along the head dimension into per-archetype buffers (Sec. 4.3) and then runs
 * each head on its own attention path (Sec. 4.4):
 *
 *   Sink    -- attends to the L keys of block 0 (the frozen sink block),
 *   Dummy   -- attends to the L keys of the current block,
 *   Spatial -- attends, in every frame of the window, to the positions within
 *              a (2r+1) x (2r+1) square around the query (clipped at borders),
 *   Global  -- attends to the whole sliding window (W blocks, current included).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  * One block holds L = frames_per_block * grid_h * grid_w tokens.  Token t of
 *    a block sits at frame f, row y, column x with t = f*grid_h*grid_w + y*grid_w + x.
 *  * q, k, v tensors are bfloat16, row-major [n_heads][tokens][head_dim], in
 *    device memory owned by the caller.  Outputs are float32 [n_heads][L][head_dim].
 *    Every device pointer must be 16-byte aligned (the kernels move 16-byte
 *    vectors); a misaligned one is HC_E_INVAL, checked before any work is queued.
 *  * A window is passed in logical order: block 0 first, then the retained
 *    blocks from oldest to newest, the current block last.  Before the window
 *    first fills (cur_block < window_blocks - 1) it holds blocks 0..cur_block.
 *  * Softmax scale s defaults to 1/sqrt(head_dim); all arithmetic on bf16
 *    inputs accumulates in float32 (QK^T and PV on the matrix cores).  Each
 *    work group first runs the softmax with its offset fixed at 0 (exact while
 *    no exponential overflows or underflows, which it checks on its row sums
 *    and accumulators) and otherwise reruns its keys as an online softmax with
 *    a running max and sum.  Partial results over key ranges are merged with
 *    their maxima and sums.
 *  * Streams: `hc_stream` is a hipStream_t (NULL = the null stream).  Work is
 *    enqueued asynchronously on it unless an entry point says otherwise.
 *  * Graph capture: once hc_attention has run on a layer at its current window
 *    fill, hc_append_block of the current block (the rewrite of a denoising
 *    step) and hc_attention only enqueue kernels on the given stream (no
 *    allocation, copy, memset or synchronisation) and may be captured into a HIP
 *    graph.  The context's host state (current block, window fill) changes when
 *    a call is made, not when a graph replays it, so a captured sequence must not
 *    advance the block; the first hc_attention at a new window fill builds the
 *    layer's work list (it allocates and synchronises) and runs eagerly.
 *  * Errors: every entry point returns an hc_status; nothing is thrown across
 *    the ABI.  On failure the context keeps a message (hc_last_error) and the
 *    layer state is left as it was before the call, with two exceptions: after
 *    HC_E_DEVICE the device memory contents of that layer are unspecified, and
 *    after HC_E_NOMEM or HC_E_DEVICE from hc_set_head_types or
 *    hc_classify_heads the layer may have no head table (its old buffers are
 *    released before the new ones are allocated, so replacing a table never
 *    needs the memory of two); it then answers HC_E_STATE until a table is set.
 *  * A context is not thread-safe; use one context per stream of work.
 */
#ifndef HEADCAST_H
#define HEADCAST_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct hc_ctx hc_ctx;
typedef void *hc_stream;   /* hipStream_t */

typedef enum {
  HC_OK = 0,
  HC_E_INVAL = -1,   /* bad argument: null pointer, bad layer, bad size, bad label   */
  HC_E_STATE = -2,   /* call not valid in the layer's current state                  */
  HC_E_ORDER = -3,   /* block index neither the current block nor the next one       */
  HC_E_NOMEM = -4,   /* device allocation failed                                      */
  HC_E_DEVICE = -5   /* a HIP runtime call failed (message in hc_last_error)          */
} hc_status;

/* Head archetypes (Sec. 3.2 observations, Sec. 4.2 decision rule). uint8 per head. */
enum { HC_SINK = 0, HC_DUMMY = 1, HC_SPATIAL = 2, HC_GLOBAL = 3 };

/* Per-head classification statistics written by hc_classify_heads (Eq. 3, Eq. 4). */
enum {
  HC_STAT_COS_SINK = 0,    /* mean token cosine of the Sink proxy vs O_ref      */
  HC_STAT_COS_DUMMY = 1,   /* mean token cosine of the Dummy proxy vs O_ref     */
  HC_STAT_COS_SPATIAL = 2, /* mean token cosine of the Spatial proxy vs O_ref   */
  HC_STAT_P5 = 3,          /* 5th percentile of the Spatial token cosines       */
  HC_STAT_MSE = 4,         /* mean squared difference O_spatial - O_ref         */
  HC_STAT_SCORE = 5,       /* P5 - gamma * MSE                                  */
  HC_N_STATS = 6
};

typedef struct {
  int32_t n_layers;          /* layers the context manages (>= 1)                      */
  int32_t n_heads;           /* heads per layer, 1..64                                 */
  int32_t head_dim;          /* 64 or 128                                              */
  int32_t grid_h, grid_w;    /* latent tokens per frame = grid_h * grid_w              */
  int32_t frames_per_block;  /* 1..4 latent frames per block (Sec. 5.1 uses 3)         */
  int32_t window_blocks;     /* W >= 2, counts the frozen sink block and the current   */
  int32_t spatial_radius;    /* r of the deployed Spatial path, 0..12                  */
  int32_t proxy_radius;      /* r_p of the classification Spatial proxy, 0..12 (Sec. 5.1: 2) */
  float theta_sink;          /* Eq. 5 thresholds (Sec. 5.1: 0.95, 0.95, 0.95, 0.755)  */
  float theta_dummy;
  float theta_spatial;
  float theta_score;
  float gamma;               /* MSE weight of Eq. 4 (Sec. 5.1: 5)                     */
  float softmax_scale;       /* 0 => 1/sqrt(head_dim)                                 */
  int32_t spatial_cell;      /* 0: Spatial heads use the centred (2r+1)^2 window (the
                              * Sec. 4.2 proxy geometry).  c in 2..64: the deployed cell
                              * variant of Sec. 4.4 -- every frame is cut into c x c
                              * cells (round(grid/c) per axis, halves rounded up, the last
                              * cell ending at the border) and a query attends to its own
                              * cell in every window frame (Sec. 5.1: c = 10).  At most 64
                              * cells per axis.  The classification proxy always uses the
                              * centred window of radius proxy_radius.                  */
  int32_t sd_blocks;         /* 1: a Sink head attends to block 0 and a Dummy head to the
                              * current block (L keys; the Sec. 4.2 proxies and the
                              * "exactly one block" of Sec. 4.4).  2: the App. B / App. C
                              * reading -- Sink to block 0 and the current block, Dummy
                              * to the previous and the current block (2L keys once a
                              * previous block exists; needs window_blocks >= 3 so that
                              * the previous block lies in the window, else
                              * HC_E_INVAL).  The classification proxies use one block
                              * either way.                                             */
} hc_config;

/* Fills the paper's defaults (Sec. 5.1) for a 30 x 12-head, head_dim 128,
 * 3-frame-block, 7-block-window model at a 30x52 latent grid, r = 4, r_p = 2.
 * Never fails. */
void hc_config_default(hc_config *cfg);

/* HC_OK if the configuration is usable, else HC_E_INVAL.  Pure host check.
 * Besides the ranges above: L = frames_per_block*grid_h*grid_w must be a
 * multiple of 8 and W*L must fit in int32. */
hc_status hc_validate_config(const hc_config *cfg);

/* Static strings, never NULL. */
const char *hc_status_string(hc_status s);
/* Message of the last failing call on ctx ("" if none); valid until the next call. */
const char *hc_last_error(const hc_ctx *ctx);

/* Physical ring slot that block `block` occupies in a Global or Spatial buffer
 * with `window_blocks` slots: slot 0 keeps block 0 for good; later blocks
 * rotate through slots 1..W-1, evicting the oldest rolling block (Sec. 4.3,
 * "sliding-window layout retaining the initial sink tokens").  Pure host
 * function; returns -1 for block < 0 or window_blocks < 2. */
int32_t hc_ring_slot(int64_t block, int32_t window_blocks);

/* Creates a context on HIP device `device`.  The context owns all per-layer
 * compact buffers, head tables and work lists; it allocates per-layer buffers
 * when head types are first set.  Returns HC_E_INVAL (bad config / null out),
 * HC_E_DEVICE (device not usable) or HC_E_NOMEM. */
hc_status hc_create(const hc_config *cfg, int device, hc_ctx **out);
void hc_destroy(hc_ctx *ctx);   /* NULL is allowed; synchronises the device first */

/* One-time online classification of one layer (Sec. 4.2, Eq. 2-5), followed by
 * the cache split (Sec. 4.3).
 *   q      : bf16 [H][L][d]   queries of the current block (device)
 *   k_win, v_win : bf16 [H][W*L][d] the full window in logical order (device)
 *   types_out : host uint8 [H]   decided archetype per head (required)
 *   stats_out : host double [H][HC_N_STATS] statistics, or NULL
 * The current block is `cur_block`; the window must be full, i.e.
 * cur_block >= W-1 (the paper fires classification when the window first
 * fills), else HC_E_STATE.  Computes O_ref and the three proxy outputs, the
 * per-token cosines and squared errors, and per head the means, P5 (exact
 * order statistics, linear interpolation at rank 0.05 (L-1)), MSE and score
 * on the GPU (statistics in float64), and the Eq. 5 decision on the host from
 * those six numbers.  Then sets the layer's head
 * table and splits k_win / v_win into the compact buffers, exactly as
 * hc_set_head_types would.  SYNCHRONISES `stream` (the labels are host
 * outputs).  Needs device memory of about 2 * H*W*L*d*2 bytes (the window in
 * Global layout) + the window in Spatial layout (rows padded to a multiple of 8
 * keys) + 4 * H*L*d*4 bytes
 * (the proxy outputs) + the per-block partials (H*W*ceil(L/128) slots of
 * 128*(d+2) floats) + the token statistics (H*L*4 doubles): the first call allocates it, the context keeps it for
 * later calls (every layer of a generation) and releases it in hc_destroy;
 * hc_memory_bytes counts it. */
hc_status hc_classify_heads(hc_ctx *ctx, int layer, int64_t cur_block, const void *q,
                            const void *k_win, const void *v_win, uint8_t *types_out,
                            double *stats_out, hc_stream stream);

/* The classification outputs of the last hc_classify_heads call on this
 * context that returned HC_OK (Sec. 4.2: Eq. 2 and the three proxies), for
 * inspection of a decision and for checking the classification attention on
 * its own.  which: HC_CLS_O_REF (attention over the full window),
 * HC_CLS_O_SINK (block 0 alone), HC_CLS_O_DUMMY (the current block alone),
 * HC_CLS_O_SPATIAL (centred window of radius proxy_radius in every window
 * frame).  dst: device float32 [H][L][d], written by a copy enqueued on
 * `stream`.  The outputs are those of the layer classified last (each call
 * overwrites them).  HC_E_STATE before a successful classification,
 * HC_E_INVAL for another `which` or a NULL or misaligned dst. */
enum {
  HC_CLS_O_REF = 0,
  HC_CLS_O_SINK = 1,
  HC_CLS_O_DUMMY = 2,
  HC_CLS_O_SPATIAL = 3
};
hc_status hc_classify_outputs(hc_ctx *ctx, int which, float *dst, hc_stream stream);

/* Sets a layer's head table without classifying (restored labels, fixed
 * tables, the all-Global full-window baseline) and splits the given window
 * (bf16 [H][n*L][d], n = min(cur_block+1, W), logical order, device) into
 * compact buffers (Sec. 4.3): Sink heads keep block 0, Dummy heads the current
 * block, Global and Spatial heads the whole window in ring slots.
 * types: host uint8 [H] with values HC_SINK..HC_GLOBAL (else HC_E_INVAL).
 * Re-setting a layer replaces its buffers.  Async on `stream` apart from
 * allocation. */
hc_status hc_set_head_types(hc_ctx *ctx, int layer, const uint8_t *types, int64_t cur_block,
                            const void *k_win, const void *v_win, hc_stream stream);

/* Layout integers of a layer (host outputs):
 *   head_slot [H] : index of each head inside its buffer; Sink and Dummy heads
 *                   share the Sink-Dummy buffer; heads keep head-id order.
 *   ring_slot_of_logical [W] : physical slot of each logical window position
 *                   (sink block first, current block last), -1 while empty.
 * Either pointer may be NULL.  HC_E_STATE if the layer has no head table. */
hc_status hc_get_layout(const hc_ctx *ctx, int layer, int32_t *head_slot,
                        int32_t *ring_slot_of_logical);

/* Writes one block's K and V (bf16 [H][L][d], device) into the layer's
 * buffers (Sec. 4.3): Global and Spatial heads into the block's ring slot,
 * Dummy heads over their single block (rolling overwrite), Sink heads only for
 * block 0.  `block` equal to the current block overwrites it (the next
 * denoising step of the same block); current + 1 advances the window and
 * evicts the oldest rolling block.  Anything else: HC_E_ORDER.  HC_E_STATE if
 * the layer has no head table.  Async. */
hc_status hc_append_block(hc_ctx *ctx, int layer, int64_t block, const void *k_blk,
                          const void *v_blk, hc_stream stream);

/* Head-specific attention of one layer over all heads (Sec. 4.4):
 *   q : bf16 [H][L][d] queries of the current block (device)
 *   head_types : host uint8 [H]; must equal the layer's table (else HC_E_STATE)
 *   o : float32 [H][L][d] (device), every head written in place.
 * Launches the grouped work of the layer: every Global head is cut into one
 * work unit per window block and every Sink/Dummy head into one unit, each
 * unit 128 queries wide, so all units of the dense kernel cost the same; the
 * per-block partial results of Global heads are merged by a combine kernel;
 * Spatial heads run on the windowed kernel (when they give too few work groups
 * to fill the GPU, their key frames are cut into ranges whose partial results
 * a merge kernel combines).  Async. */
hc_status hc_attention(hc_ctx *ctx, int layer, const void *q, const uint8_t *head_types,
                       float *o, hc_stream stream);

/* Bytes of the fixed device scratch that hc_attention_static works in. */
#define HC_STATIC_SCRATCH_BYTES (64u << 20)

/* hc_attention for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation.  Same
 * arguments, head table check and outputs as hc_attention (within its
 * floating-point tolerance: the work is not tail-balanced, so partial results
 * may be merged in another order).  It allocates nothing, copies nothing from
 * the host and does not synchronise: the layer's work list, the per-block
 * partial results of Global (and two-block Sink/Dummy) heads and the split
 * partials of Spatial heads live in one fixed array of HC_STATIC_SCRATCH_BYTES
 * per GPU, held by the library until the process ends; the work list is
 * written by a kernel on `stream` at every call.  Every call on a GPU uses
 * that GPU's array and leaves its contents behind, so calls that overlap on
 * one GPU (other streams, other contexts, other threads) race and must be
 * ordered by the caller.  A layer whose work needs more than the array holds
 * (the Spatial split is dropped first) is HC_E_INVAL with the size in
 * hc_last_error, before anything is enqueued; so is a context with the cell
 * variant (spatial_cell > 0).  The layer's buffers are the context's, set up
 * beforehand by hc_set_head_types / hc_classify_heads. */
hc_status hc_attention_static(hc_ctx *ctx, int layer, const void *q, const uint8_t *head_types,
                              float *o, hc_stream stream);

/* Device bytes held by the context's buffers (all layers, partial-result
 * slots, and the classification memory once hc_classify_heads has run). */
hc_status hc_memory_bytes(const hc_ctx *ctx, int64_t *bytes);

/* Kernel timing: when enabled, every launch the context makes records a pair
 * of HIP events on the stream it is launched on.  hc_profile_read synchronises
 * those events and returns the summed duration (ms) and the launch count of
 * one kernel kind since the last reset, then resets it. */
enum { HC_K_DENSE = 0, HC_K_SPATIAL = 1, HC_K_SCATTER = 2, HC_K_STATS = 3, HC_K_COMBINE = 4,
       HC_K_COUNT = 5 };
hc_status hc_profile_enable(hc_ctx *ctx, int on);
hc_status hc_profile_read(hc_ctx *ctx, int kernel_kind, double *total_ms, int64_t *launches);

#ifdef __cplusplus
}
#endif
#endif /* HEADCAST_H */
