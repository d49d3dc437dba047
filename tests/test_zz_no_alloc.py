"""hc_attention_static, the routed layer-step for callers that cannot allocate
device memory, against hc_attention on the same context and inputs (through
the C ABI): two calls in a row on the static entry point, the second on a
smaller layer, each compared with the allocating entry point within the
output tolerance (max-abs 1e-2, mean-abs 1e-3); a layer whose work does not
fit the fixed scratch is rejected before anything runs."""
import numpy as np
import pytest

from helpers import MAX_ABS, MEAN_ABS
from synth import inputs as S

pytestmark = pytest.mark.gpu


def _layer(hc, w, types, seed, cfg_kw=None):
    import torch
    H, L, d, W = w.n_heads, w.block_tokens, w.head_dim, w.window_blocks
    dev = torch.device("cuda:0")
    ctx = hc.Context(hc.config_from_workload(w, n_layers=1, **(cfg_kw or {})), 0)
    kw = S.device_normal_bf16((H, W * L, d), seed, dev)
    vw = S.device_normal_bf16((H, W * L, d), seed + 1, dev)
    ctx.set_head_types(0, types, W - 1, kw, vw)
    q = S.device_normal_bf16((H, L, d), seed + 2, dev)
    return ctx, q


def _compare(got, ref, what):
    err = (got.double() - ref.double()).abs()
    mx, mean = err.max().item(), err.mean().item()
    print(f"{what}: max|static - hc_attention| {mx:.3e} mean {mean:.3e}", flush=True)
    assert bool(got.isfinite().all()), what
    assert mx <= MAX_ABS and mean <= MEAN_ABS, (what, mx, mean)


def test_static_entry_point_two_calls_then_smaller(hc):
    import torch
    # call 1: a 480P-shaped layer (L = 4680, 7-block window) with one Global head
    # (7 partials per query tile), two Spatial heads (split over key frames) and
    # nine Sink/Dummy heads; call 2: the tiny layer (L = 128), smaller in every
    # dimension, on the same GPU's scratch
    w1 = S.WORKLOADS["480p"].scaled(n_layers=1)
    t1 = np.array([3, 2, 0, 1, 2, 0, 1, 0, 1, 0, 1, 0], np.uint8)
    w2 = S.WORKLOADS["tiny"]
    t2 = S.head_types(w2)[0]
    cases = [("480P layer", w1, t1, 11), ("tiny layer", w2, t2, 21)]
    ctxs = []
    for what, w, t, seed in cases:
        print(f"static entry point: {what}", flush=True)
        ctx, q = _layer(hc, w, t, seed)
        ctxs.append(ctx)
        shape = (w.n_heads, w.block_tokens, w.head_dim)
        ref = torch.full(shape, float("nan"), dtype=torch.float32, device="cuda")
        got = torch.full(shape, float("nan"), dtype=torch.float32, device="cuda")
        ctx.attention(0, q, t, ref)
        ctx.attention_static(0, q, t, got)
        torch.cuda.synchronize()
        _compare(got, ref, what)
    for c in ctxs:
        c.close()


def test_static_entry_point_two_block_variant(hc):
    import torch
    # two Sink-Dummy slots: every Sink/Dummy head merges two block partials
    w = S.WORKLOADS["tiny"].scaled(window_blocks=4)
    t = S.head_types(w)[0]
    ctx, q = _layer(hc, w, t, 31, {"sd_blocks": 2})
    shape = (w.n_heads, w.block_tokens, w.head_dim)
    ref = torch.empty(shape, dtype=torch.float32, device="cuda")
    got = torch.full(shape, float("nan"), dtype=torch.float32, device="cuda")
    ctx.attention(0, q, t, ref)
    ctx.attention_static(0, q, t, got)
    torch.cuda.synchronize()
    _compare(got, ref, "two-block Sink/Dummy")
    ctx.close()


def test_static_entry_point_rejects_oversized_layer(hc):
    import torch
    # a 720P layer of twelve Global heads needs 12 x 85 x 7 partial slots of
    # 128 x 130 floats: far beyond the fixed scratch
    w = S.WORKLOADS["720p"].scaled(n_layers=1)
    t = np.full(w.n_heads, S.GLOBAL, np.uint8)
    ctx, q = _layer(hc, w, t, 41)
    o = torch.full((w.n_heads, w.block_tokens, w.head_dim), float("nan"), dtype=torch.float32,
                   device="cuda")
    with pytest.raises(hc.HeadCastError) as e:
        ctx.attention_static(0, q, t, o)
    assert e.value.status == hc.HC_E_INVAL and "needs" in str(e.value)
    torch.cuda.synchronize()
    assert bool(o.isnan().all())          # nothing was enqueued
    ctx.close()
