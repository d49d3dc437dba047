"""The autoregressive schedule (paper_2607_20125_amd.ar_loop): full-window
attention while the window fills, classification at the first denoising step of
the block that fills it, then routed attention with per-step overwrites and
block advances.  Tiny planted workload, two layers, two denoising steps per
block.  The first step of a block carries its own K and V (channel 0 of K and
all of V drawn afresh; the planted structure untouched), the last step the
block's final values, so every output checked below depends on the last step
having overwritten the first in every buffer.  The labels must be the planted
ones and the oracle's on the window the classification saw (earlier blocks
at their last step, the current block at its first), and the outputs of the
last step of every block must match the oracle on the final window."""
import numpy as np
import pytest

from helpers import assert_close, dev_bf16, out_tensor
from oracle import headcast_oracle as O
from synth import inputs as S

pytestmark = pytest.mark.gpu


def test_tiny_planted_ar_loop(hc):
    from paper_2607_20125_amd import ar_loop

    w = S.WORKLOADS["tiny_planted"].scaled(n_layers=2, mix=(2, 2, 2, 2))
    W = w.window_blocks
    n_blocks = W + 3
    ctx = hc.Context(hc.config_from_workload(w), 0)
    cache = {}

    def first_step(layer, b):
        """K and V of a block's first denoising step (bf16 bits)."""
        _, k, v = S.gen_step_block(w, layer, b, classify_block=W - 1)
        rng = np.random.default_rng([w.seed, layer, b, 99])
        kf = S.bf16_bits_to_f32(k).copy()
        kf[:, :, 0] = rng.standard_normal(kf.shape[:2], dtype=np.float32)
        vf = rng.standard_normal(v.shape, dtype=np.float32)
        return S.f32_to_bf16_bits(kf), S.f32_to_bf16_bits(vf)

    def block_data(layer, b, si):
        if (layer, b) not in cache:
            q, k, v = S.gen_step_block(w, layer, b, classify_block=W - 1)
            k0, v0 = first_step(layer, b)
            cache[(layer, b)] = (dev_bf16(q), dev_bf16(k), dev_bf16(v), q, dev_bf16(k0),
                                 dev_bf16(v0), k0, v0)
        c = cache[(layer, b)]
        return (c[0], c[4], c[5]) if si == 0 else (c[0], c[1], c[2])

    out = out_tensor(w)
    seen = {}

    def on_step(layer, b, si, types, q):
        if si == 1:
            seen[(layer, b)] = (out.cpu().numpy(), np.array(types))

    res = ar_loop.run(ctx, n_blocks, block_data, out, steps=(1000, 750), on_step=on_step)
    assert res.classified_at == W - 1 and res.classify_ms > 0
    L = w.block_tokens
    for layer in range(w.n_layers):
        assert list(res.types[layer]) == list(S.head_types(w)[layer])
        # the window at the classification: blocks 0 .. W-2 as their last step
        # wrote them, block W-1 at its first step
        _, kw, vw = S.gen_layer(w, layer, W - 1, classify_block=W - 1)
        kw, vw = kw.copy(), vw.copy()
        kw[:, (W - 1) * L:] = cache[(layer, W - 1)][6]
        vw[:, (W - 1) * L:] = cache[(layer, W - 1)][7]
        q0 = cache[(layer, W - 1)][3]
        ref_labels, _ = O.classify_layer(q0, kw, vw, w.grid_h, w.grid_w, w.frames_per_block,
                                         w.proxy_radius)
        assert list(res.types[layer]) == list(ref_labels)
    for (layer, b), (got, types) in sorted(seen.items()):
        expect = np.full(w.n_heads, S.GLOBAL) if b < W - 1 else S.head_types(w)[layer]
        assert list(types) == list(expect)
        _, kw, vw = S.gen_layer(w, layer, b, classify_block=W - 1)
        ref = O.routed_attention(types, cache[(layer, b)][3], kw, vw, w.grid_h, w.grid_w,
                                 w.frames_per_block, w.spatial_radius)
        assert_close(got, ref, f"AR loop layer {layer} block {b}")
    assert len(res.ms_per_block) == n_blocks
