"""GPU parity: the HIP path (called through the C ABI) against the CPU oracle on
the same seeded bf16 inputs.  Attention outputs: max-abs 1e-2 and mean-abs 1e-3;
labels and layout integers: bit-exact."""
import numpy as np
import pytest

from helpers import assert_close, dev_bf16, out_tensor, stratified_rows
from oracle import headcast_oracle as O
from synth import inputs as S

pytestmark = pytest.mark.gpu


def oracle_layer(w, types, q, k, v, rows=None, r=None):
    return O.routed_attention(types, q, k, v, w.grid_h, w.grid_w, w.frames_per_block,
                              w.spatial_radius if r is None else r, rows=rows)


def gpu_layer(hc, w, types, cur, q, k, v, ctx=None):
    import torch
    ctx = ctx or hc.Context(hc.config_from_workload(w, n_layers=1), 0)
    ctx.set_head_types(0, types, cur, dev_bf16(k), dev_bf16(v))
    o = out_tensor(w)
    ctx.attention(0, dev_bf16(q), types, o)
    torch.cuda.synchronize()
    return ctx, o.cpu().numpy()


# --- tiny: full tensors ------------------------------------------------------------------
@pytest.mark.parametrize("cur", [0, 1, 3, 6])
def test_tiny_fixed_table(hc, cur):
    w = S.WORKLOADS["tiny"]
    types = S.head_types(w)[0]
    q, k, v = S.gen_layer(w, 0, cur)
    print(f"tiny fixed table cur_block={cur}", flush=True)
    _, got = gpu_layer(hc, w, types, cur, q, k, v)
    assert_close(got, oracle_layer(w, types, q, k, v), f"tiny cur={cur}")


@pytest.mark.parametrize("kind", [S.SINK, S.DUMMY, S.SPATIAL, S.GLOBAL])
def test_tiny_homogeneous(hc, kind):
    w = S.WORKLOADS["tiny"]
    types = np.full(4, kind, np.uint8)
    q, k, v = S.gen_layer(w, 0, 5)
    print(f"tiny homogeneous kind={kind}", flush=True)
    _, got = gpu_layer(hc, w, types, 5, q, k, v)
    assert_close(got, oracle_layer(w, types, q, k, v), f"tiny all-{S.TYPE_NAMES[kind]}")


@pytest.mark.parametrize("r", [0, 2, 3, 4, 5, 7])
def test_tiny_spatial_radii(hc, r):
    w = S.WORKLOADS["tiny"].scaled(spatial_radius=r)
    types = np.full(4, S.SPATIAL, np.uint8)
    q, k, v = S.gen_layer(w, 0, 3)
    print(f"tiny spatial r={r}", flush=True)
    _, got = gpu_layer(hc, w, types, 3, q, k, v)
    assert_close(got, oracle_layer(w, types, q, k, v), f"tiny spatial r={r}")
    if r >= max(w.grid_h, w.grid_w) - 1:     # the window covers the frame: Global
        glob = oracle_layer(w, np.full(4, S.GLOBAL, np.uint8), q, k, v)
        assert_close(got, glob, "spatial covering the frame vs Global")


def test_tiny_ragged_grid(hc):
    # 5 x 8 frame, 1 frame per block, head_dim 128: ragged column tiles and query tiles
    w = S.Workload("ragged", 1, 6, 128, 5, 8, 1, 3, 2, 2, 11, (1, 2, 2, 1))
    types = np.array([3, 2, 0, 1, 2, 3], np.uint8)
    for cur in (1, 2, 4):
        q, k, v = S.gen_layer(w, 0, cur)
        _, got = gpu_layer(hc, w, types, cur, q, k, v)
        assert_close(got, oracle_layer(w, types, q, k, v), f"ragged cur={cur}")


def test_grid_width_not_multiple_of_8(hc):
    # 480P-like row pitch (13 -> padded to 16) on a small grid: 4 x 13 frame, 2 frames
    w = S.Workload("pitch", 1, 4, 128, 4, 13, 2, 4, 4, 2, 13, (1, 1, 1, 1))   # L = 104
    types = np.array([2, 3, 2, 1], np.uint8)
    q, k, v = S.gen_layer(w, 0, 3)
    _, got = gpu_layer(hc, w, types, 3, q, k, v)
    assert_close(got, oracle_layer(w, types, q, k, v), "pitch 13")


@pytest.mark.parametrize("cur", [31, 40])
def test_largest_window_and_frames(hc, cur):
    # W = 32 window blocks (the largest: every Global merge has 32 partial slots) and
    # F = 4 frames per block (four waves per Spatial work group), r = 12, head_dim 64
    w = S.Workload("maxwin", 1, 4, 64, 8, 8, 4, 32, 12, 2, 32, (1, 1, 1, 1))   # L = 256
    types = np.array([0, 1, 2, 3], np.uint8)
    print(f"largest window W=32 F=4 cur_block={cur}", flush=True)
    q, k, v = S.gen_layer(w, 0, cur)
    _, got = gpu_layer(hc, w, types, cur, q, k, v)
    assert_close(got, oracle_layer(w, types, q, k, v), f"W=32 F=4 cur={cur}")


def test_largest_head_count(hc):
    # 64 heads (the largest), 16 of each type in a seeded order: head ids up to 63 in
    # every work list, slots up to 31 in the shared Sink-Dummy buffer
    w = S.Workload("h64", 1, 64, 64, 8, 8, 2, 4, 1, 2, 64, (16, 16, 16, 16))
    types = S.head_types(w)[0]
    assert sorted(np.bincount(types, minlength=4)) == [16, 16, 16, 16]
    q, k, v = S.gen_layer(w, 0, 5)
    ctx, got = gpu_layer(hc, w, types, 5, q, k, v)
    assert_close(got, oracle_layer(w, types, q, k, v), "64 heads")
    hs, _ = ctx.get_layout(0)
    assert list(hs) == O.head_slots(types)


@pytest.mark.parametrize("hg,wg,f", [(1, 8, 1), (8, 1, 1), (2, 2, 2), (1, 2, 4)])
@pytest.mark.parametrize("cur", [0, 4])
def test_degenerate_grids(hc, hg, wg, f, cur):
    # the smallest blocks the ABI accepts (8 tokens): a single row, a single column,
    # a 2 x 2 grid, a 1 x 2 grid over 4 frames; every tile is mostly padding and every
    # Spatial halo is clipped on all sides
    w = S.Workload("degen", 1, 4, 64, hg, wg, f, 3, 2, 1, 7, (1, 1, 1, 1))
    types = np.array([0, 1, 2, 3], np.uint8)
    print(f"degenerate grid {hg}x{wg} F={f} cur_block={cur}", flush=True)
    q, k, v = S.gen_layer(w, 0, cur)
    _, got = gpu_layer(hc, w, types, cur, q, k, v)
    assert_close(got, oracle_layer(w, types, q, k, v), f"grid {hg}x{wg} F={f} cur={cur}")


@pytest.mark.parametrize("scale", [0.05, 0.3])
def test_custom_softmax_scale(hc, scale):
    # a softmax scale other than 1/sqrt(d) reaches every path (dense and Spatial)
    import torch
    w = S.WORKLOADS["tiny"]
    types = S.head_types(w)[0]
    cur = 5
    q, k, v = S.gen_layer(w, 0, cur)
    cfg = hc.config_from_workload(w, n_layers=1)
    cfg.softmax_scale = scale
    ctx = hc.Context(cfg, 0)
    ctx.set_head_types(0, types, cur, dev_bf16(k), dev_bf16(v))
    o = out_tensor(w)
    ctx.attention(0, dev_bf16(q), types, o)
    torch.cuda.synchronize()
    ref = O.routed_attention(types, q, k, v, w.grid_h, w.grid_w, w.frames_per_block,
                             w.spatial_radius, scale=scale)
    assert_close(o.cpu().numpy(), ref, f"softmax scale {scale}")


# --- ring buffer across appends, overwrite and eviction ---------------------------------------
def test_tiny_append_ring_wrap(hc):
    import torch
    w = S.WORKLOADS["tiny"]
    W = w.window_blocks
    types = S.head_types(w)[0]
    ctx = hc.Context(hc.config_from_workload(w), 0)
    cur = W - 1
    q, k, v = S.gen_layer(w, 0, cur)
    ctx.set_head_types(0, types, cur, dev_bf16(k), dev_bf16(v))
    other = w.scaled(seed=99)
    for b in range(W, 3 * W + 2):
        # first a stale write of block b (another seed), then the real one (overwrite)
        _, kb0, vb0 = S.gen_step_block(other, 0, b)
        ctx.append_block(0, b, dev_bf16(kb0), dev_bf16(vb0))
        qb, kb, vb = S.gen_step_block(w, 0, b)
        ctx.append_block(0, b, dev_bf16(kb), dev_bf16(vb))
        o = out_tensor(w)
        ctx.attention(0, dev_bf16(qb), types, o)
        torch.cuda.synchronize()
        _, kw, vw = S.gen_layer(w, 0, b)
        assert_close(o.cpu().numpy(), oracle_layer(w, types, qb, kw, vw), f"append b={b}")
        hs, ring = ctx.get_layout(0)
        assert list(ring) == O.ring_slots_of_logical(b, W)
        assert list(hs) == O.head_slots(types)


def test_tiny_warmup_appends_before_window_fills(hc):
    import torch
    w = S.WORKLOADS["tiny"]
    types = np.array([3, 2, 1, 0], np.uint8)
    ctx = hc.Context(hc.config_from_workload(w), 0)
    q, k, v = S.gen_layer(w, 0, 0)
    ctx.set_head_types(0, types, 0, dev_bf16(k), dev_bf16(v))
    for b in range(1, 2 * w.window_blocks):
        qb, kb, vb = S.gen_step_block(w, 0, b)
        ctx.append_block(0, b, dev_bf16(kb), dev_bf16(vb))
        o = out_tensor(w)
        ctx.attention(0, dev_bf16(qb), types, o)
        torch.cuda.synchronize()
        _, kw, vw = S.gen_layer(w, 0, b)
        assert_close(o.cpu().numpy(), oracle_layer(w, types, qb, kw, vw), f"warm-up b={b}")
        assert list(ctx.get_layout(0)[1]) == O.ring_slots_of_logical(b, w.window_blocks)


# --- fingerprint: Q = 0 gives exact means of integer-valued V ------------------------------
def test_fingerprint_key_sets_and_ring(hc):
    import torch
    w = S.WORKLOADS["tiny"].scaled(spatial_radius=2)
    W, L, P, Wg, F = w.window_blocks, w.block_tokens, w.tokens_per_frame, w.grid_w, w.frames_per_block
    types = S.head_types(w)[0]
    ctx = hc.Context(hc.config_from_workload(w), 0)
    cur = 9
    ids = S.window_block_ids(cur, W)
    # V columns: 1, y', x', frame-in-block, block id, (block id % 5); rest 0.  bf16-exact.
    def vblock(b):
        t = np.arange(L)
        cols = np.zeros((L, w.head_dim), np.float32)
        cols[:, 0] = 1
        cols[:, 1] = (t % P) // Wg
        cols[:, 2] = (t % P) % Wg
        cols[:, 3] = t // P
        cols[:, 4] = b
        cols[:, 5] = b % 5
        return S.f32_to_bf16_bits(np.broadcast_to(cols, (w.n_heads, L, w.head_dim)).copy())
    kz = S.f32_to_bf16_bits(np.random.default_rng(0).standard_normal(
        (w.n_heads, L, w.head_dim)).astype(np.float32))
    k = np.concatenate([kz] * len(ids), axis=1)
    v = np.concatenate([vblock(b) for b in ids], axis=1)
    q = np.zeros((w.n_heads, L, w.head_dim), np.uint16)
    ctx.set_head_types(0, types, cur, dev_bf16(k), dev_bf16(v))
    o = out_tensor(w)
    ctx.attention(0, dev_bf16(q), types, o)
    torch.cuda.synchronize()
    got = o.cpu().numpy()
    ref = oracle_layer(w, types, q, k, v)
    np.testing.assert_allclose(got, ref, atol=2e-5, rtol=0)
    # closed forms: Sink sees block 0 only, Dummy the current block only
    np.testing.assert_allclose(got[0, :, 4], 0.0, atol=1e-6)
    np.testing.assert_allclose(got[1, :, 4], cur, atol=1e-5)
    np.testing.assert_allclose(got[3, :, 4], np.mean(ids), atol=1e-5)


# --- Wan-shaped layers ---------------------------------------------------------------------------
def test_480p_full_layer(hc):
    w = S.WORKLOADS["480p"]
    types = S.head_types(w)[0]
    cur = w.window_blocks - 1
    print("480p layer 0 generate", flush=True)
    q, k, v = S.gen_layer(w, 0, cur)
    print("480p layer 0 gpu", flush=True)
    _, got = gpu_layer(hc, w, types, cur, q, k, v)
    print("480p layer 0 oracle", flush=True)
    assert_close(got, oracle_layer(w, types, q, k, v), "480p layer 0")


@pytest.mark.parametrize("name", ["720p", "1080p"])
def test_sampled_rows(hc, name):
    w = S.WORKLOADS[name]
    layer = 1
    types = S.head_types(w)[layer]
    cur = w.window_blocks - 1
    print(f"{name} layer {layer} generate", flush=True)
    q, k, v = S.gen_layer(w, layer, cur)
    print(f"{name} gpu", flush=True)
    _, got = gpu_layer(hc, w, types, cur, q, k, v)
    rows = stratified_rows(w)
    print(f"{name} oracle on {rows.size} rows x {w.n_heads} heads", flush=True)
    assert_close(got[:, rows], oracle_layer(w, types, q, k, v, rows=rows), f"{name} sampled")


def test_480p_shape_head_dim_64_sampled(hc):
    """The head_dim 64 kernels at a Wan-sized layer (480P grid and window, twelve
    64-dim heads, the 480P head mix of layer 2), on stratified rows."""
    base = S.WORKLOADS["480p"]
    w = S.Workload("480p_d64", 1, base.n_heads, 64, base.grid_h, base.grid_w,
                   base.frames_per_block, base.window_blocks, base.spatial_radius,
                   base.proxy_radius, 6464, (3, 3, 3, 3))
    types = S.head_types(base)[2]
    cur = w.window_blocks - 1
    q, k, v = S.gen_layer(w, 0, cur)
    _, got = gpu_layer(hc, w, types, cur, q, k, v)
    rows = stratified_rows(w)
    assert_close(got[:, rows], oracle_layer(w, types, q, k, v, rows=rows), "480p d=64 sampled")


def test_720p_all_global_baseline_sampled(hc):
    w = S.WORKLOADS["720p"]
    types = np.full(w.n_heads, S.GLOBAL, np.uint8)
    cur = w.window_blocks - 1
    q, k, v = S.gen_layer(w, 2, cur, heads=range(w.n_heads))
    _, got = gpu_layer(hc, w, types, cur, q, k, v)
    rows = stratified_rows(w, n_random=256, seed=1)
    assert_close(got[:, rows], oracle_layer(w, types, q, k, v, rows=rows), "720p full-window")


# Spatial work split over key frames (few Spatial heads) and not split (many),
# also while the window is still filling (the split is capped by the valid frames)
@pytest.mark.parametrize("name,n_sp,cur", [("720p", 1, 6), ("720p", 12, 6), ("480p", 1, 1),
                                           ("480p", 2, 6)])
def test_spatial_split_paths(hc, name, n_sp, cur):
    w = S.WORKLOADS[name]
    types = np.array([S.SPATIAL] * n_sp + [S.SINK] * (w.n_heads - n_sp), np.uint8)
    print(f"{name} {n_sp} spatial heads, block {cur}: generate", flush=True)
    q, k, v = S.gen_layer(w, 3, cur, heads=range(w.n_heads))
    _, got = gpu_layer(hc, w, types, cur, q, k, v)
    rows = stratified_rows(w, n_random=128, seed=n_sp)
    heads = list(range(n_sp))
    print(f"{name} oracle on {rows.size} rows x {n_sp} heads", flush=True)
    ref = oracle_layer(w, types, q, k, v, rows=rows)
    assert_close(got[heads][:, rows], ref[heads], f"{name} spatial x{n_sp} block {cur}")


# --- classification --------------------------------------------------------------------------------
def test_tiny_planted_classification(hc):
    import torch
    w = S.WORKLOADS["tiny_planted"]
    cur = w.window_blocks - 1
    q, k, v = S.gen_layer(w, 0, cur)
    ctx = hc.Context(hc.config_from_workload(w), 0)
    labels, stats = ctx.classify_heads(0, cur, dev_bf16(q), dev_bf16(k), dev_bf16(v))
    ref_labels, ref_stats = O.classify_layer(q, k, v, w.grid_h, w.grid_w, w.frames_per_block,
                                             w.proxy_radius)
    print("labels", labels, "stats", stats, "oracle", ref_stats, flush=True)
    assert list(labels) == list(ref_labels) == list(S.head_types(w)[0])
    np.testing.assert_allclose(stats[:, :4], ref_stats[:, :4], atol=2e-3)
    np.testing.assert_allclose(stats[:, 4], ref_stats[:, 4], rtol=2e-2, atol=1e-6)
    # the split that followed the classification serves attention for the next blocks
    for b in range(cur + 1, cur + 5):
        qb, kb, vb = S.gen_step_block(w, 0, b)
        ctx.append_block(0, b, dev_bf16(kb), dev_bf16(vb))
        o = out_tensor(w)
        ctx.attention(0, dev_bf16(qb), labels, o)
        torch.cuda.synchronize()
        _, kw, vw = S.gen_layer(w, 0, b)
        assert_close(o.cpu().numpy(), oracle_layer(w, labels, qb, kw, vw), f"post-classify b={b}")


@pytest.mark.parametrize("variant", [{"spatial_cell": 4}, {"sd_blocks": 2}])
def test_classification_in_variant_contexts(hc, variant):
    """The classification proxies are one block and the centred window whatever the
    context's paths: labels and statistics equal those of a default context, and the
    routed blocks after it follow the variant's key sets."""
    import torch
    w = S.WORKLOADS["tiny_planted"]
    cur = w.window_blocks - 1
    q, k, v = S.gen_layer(w, 0, cur)
    ref_ctx = hc.Context(hc.config_from_workload(w), 0)
    ref_labels, ref_stats = ref_ctx.classify_heads(0, cur, dev_bf16(q), dev_bf16(k), dev_bf16(v))
    ctx = hc.Context(hc.config_from_workload(w, **variant), 0)
    labels, stats = ctx.classify_heads(0, cur, dev_bf16(q), dev_bf16(k), dev_bf16(v))
    assert list(labels) == list(ref_labels)
    np.testing.assert_array_equal(stats, ref_stats)
    for b in range(cur + 1, cur + 3):
        qb, kb, vb = S.gen_step_block(w, 0, b)
        ctx.append_block(0, b, dev_bf16(kb), dev_bf16(vb))
        o = out_tensor(w)
        ctx.attention(0, dev_bf16(qb), labels, o)
        torch.cuda.synchronize()
        _, kw, vw = S.gen_layer(w, 0, b)
        ref = O.routed_attention(labels, qb, kw, vw, w.grid_h, w.grid_w, w.frames_per_block,
                                 w.spatial_radius, **variant)
        assert_close(o.cpu().numpy(), ref, f"{variant} post-classify b={b}")


def test_unbiased_tiny_classification_matches_oracle(hc):
    w = S.WORKLOADS["tiny"]
    cur = 5
    q, k, v = S.gen_layer(w, 0, cur)
    ctx = hc.Context(hc.config_from_workload(w), 0)
    labels, stats = ctx.classify_heads(0, cur, dev_bf16(q), dev_bf16(k), dev_bf16(v))
    ref_labels, ref_stats = O.classify_layer(q, k, v, w.grid_h, w.grid_w, w.frames_per_block,
                                             w.proxy_radius)
    assert list(labels) == list(ref_labels)
    np.testing.assert_allclose(stats[:, :4], ref_stats[:, :4], atol=2e-3)


# --- error paths that need a context on the device --------------------------------------------------
def test_state_and_order_errors(hc):
    w = S.WORKLOADS["tiny"]
    types = S.head_types(w)[0]
    ctx = hc.Context(hc.config_from_workload(w), 0)
    q, k, v = S.gen_layer(w, 0, 3)
    o = out_tensor(w)
    with pytest.raises(hc.HeadCastError) as e:
        ctx.attention(0, dev_bf16(q), types, o)          # no head table yet
    assert e.value.status == hc.HC_E_STATE
    with pytest.raises(hc.HeadCastError) as e:
        ctx.append_block(0, 0, dev_bf16(k[:, :w.block_tokens].copy()),
                         dev_bf16(v[:, :w.block_tokens].copy()))
    assert e.value.status == hc.HC_E_STATE
    _, k1, v1 = S.gen_layer(w, 0, 1)
    with pytest.raises(hc.HeadCastError) as e:        # window not full
        ctx.classify_heads(0, 1, dev_bf16(q), dev_bf16(np.concatenate([k1, k1], 1)),
                           dev_bf16(np.concatenate([v1, v1], 1)))
    assert e.value.status == hc.HC_E_STATE
    ctx.set_head_types(0, types, 3, dev_bf16(k), dev_bf16(v))
    wrong = types.copy(); wrong[0] = S.GLOBAL
    with pytest.raises(hc.HeadCastError) as e:
        ctx.attention(0, dev_bf16(q), wrong, o)
    assert e.value.status == hc.HC_E_STATE
    kb = dev_bf16(k[:, :w.block_tokens].copy())
    for bad in (2, 5, -1):
        with pytest.raises(hc.HeadCastError) as e:
            ctx.append_block(0, bad, kb, kb)
        assert e.value.status == hc.HC_E_ORDER
    with pytest.raises(hc.HeadCastError) as e:
        ctx.attention(1, dev_bf16(q), types, o)       # layer out of range
    assert e.value.status == hc.HC_E_INVAL
    bad_types = types.copy(); bad_types[2] = 7
    with pytest.raises(hc.HeadCastError) as e:
        ctx.attention(0, dev_bf16(q), bad_types, o)
    assert e.value.status == hc.HC_E_INVAL
    ctx.append_block(0, 3, kb, kb)      # overwrite of the current block is fine
    ctx.append_block(0, 4, kb, kb)      # so is the next block


def test_misaligned_pointers_rejected_before_any_work(hc):
    """Every device pointer must be 16-byte aligned: an offset view is HC_E_INVAL, and the
    layer keeps its state (a following call still matches the oracle)."""
    import torch
    w = S.WORKLOADS["tiny"]
    types = S.head_types(w)[0]
    ctx = hc.Context(hc.config_from_workload(w), 0)
    q, k, v = S.gen_layer(w, 0, 3)

    def shifted(a, dtype, elems):
        # the same values at an address `elems` elements past an aligned allocation
        t = a if isinstance(a, torch.Tensor) else dev_bf16(a)
        buf = torch.empty(t.numel() + elems, dtype=dtype, device=t.device)
        view = buf[elems:].view(t.shape)
        view.copy_(t)
        assert view.data_ptr() % 16 != 0 and view.is_contiguous()
        return view

    bf = torch.bfloat16
    with pytest.raises(hc.HeadCastError) as e:
        ctx.set_head_types(0, types, 3, shifted(k, bf, 1), dev_bf16(v))
    assert e.value.status == hc.HC_E_INVAL
    with pytest.raises(hc.HeadCastError) as e:
        ctx.classify_heads(0, 3, dev_bf16(q), dev_bf16(k), shifted(v, bf, 4))
    assert e.value.status == hc.HC_E_INVAL
    ctx.set_head_types(0, types, 3, dev_bf16(k), dev_bf16(v))
    kb = dev_bf16(k[:, -w.block_tokens:].copy())
    vb = dev_bf16(v[:, -w.block_tokens:].copy())
    with pytest.raises(hc.HeadCastError) as e:
        ctx.append_block(0, 3, kb, shifted(vb, bf, 2))
    assert e.value.status == hc.HC_E_INVAL
    o = out_tensor(w)
    with pytest.raises(hc.HeadCastError) as e:
        ctx.attention(0, shifted(q, bf, 3), types, o)
    assert e.value.status == hc.HC_E_INVAL
    with pytest.raises(hc.HeadCastError) as e:
        ctx.attention(0, dev_bf16(q), types, shifted(o, torch.float32, 1))
    assert e.value.status == hc.HC_E_INVAL
    ctx.append_block(0, 3, kb, vb)       # the current block rewritten with the same values
    ctx.attention(0, dev_bf16(q), types, o)
    torch.cuda.synchronize()
    ref = O.routed_attention(types, q, k, v, w.grid_h, w.grid_w, w.frames_per_block,
                             w.spatial_radius)
    assert_close(o.cpu().numpy(), ref, "after rejected calls")
