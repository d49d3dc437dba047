"""Autoregressive schedule of HeadCast over one context (Sec. 4.1 and Sec. 5.1).

A video is generated block by block; every block is denoised in a few steps
(t = 1000, 750, 500, 250 in Sec. 5.1), and every step runs attention in every
layer against the sliding window.  HeadCast's schedule on top of that:

* before the window first fills, every head attends to the whole window (the
  head table is all Global);
* at the first step (t = 1000) of the block that fills the window, each layer
  classifies its heads once (`hc_classify_heads`, which also splits the cache);
* from then on every step of every layer runs the routed paths; the first step
  of a block advances the cache, the later steps overwrite the block in place.

`run` drives that schedule through the C ABI for synthetic blocks supplied by
the caller (there is no model here: the block's Q, K and V stand in for the
projections of the denoised latents) and times each phase on the stream.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import headcast as hc

TIMESTEPS = (1000, 750, 500, 250)   # Sec. 5.1: four denoising steps per block


@dataclass
class LoopResult:
    types: list                                      # per layer: head table in force at the end
    stats: list                                      # per layer: statistics of the classification
    ms_per_block: list = field(default_factory=list)  # attention (+ appends) per block, all steps
    classify_ms: float = 0.0                         # all layers, one-time
    classified_at: int = -1                          # block index of the classification


def run(ctx: hc.Context, n_blocks: int, block_data, out, steps=TIMESTEPS, classify=True,
        on_step=None, tables_at_fill=None) -> LoopResult:
    """Runs `n_blocks` blocks of `len(steps)` denoising steps over every layer.

    block_data(layer, block, step) -> (q, k, v): bf16 device tensors [H][L][d]
        of that block at that denoising step; the cache keeps what the last
        step of a block wrote.
    out: float32 device tensor [H][L][d], reused as the output of every call.
    on_step(layer, block, step, types, q): called after each attention (tests).
    Classification fires at the first step of block W-1 when `classify`;
    otherwise the head table stays all Global (the full-window schedule), or,
    when `tables_at_fill` (per layer) is given, those tables are installed at
    that point instead of classifying (a table decided offline).
    """
    import torch

    cfg = ctx.cfg
    H, W, NL = cfg.n_heads, cfg.window_blocks, cfg.n_layers
    all_g = np.full(H, hc.GLOBAL, np.uint8)
    types = [all_g.copy() for _ in range(NL)]
    stats = [None] * NL
    # the blocks before the classification block as their last step wrote them,
    # to hand the full window to the classification call in logical order
    held_k = [dict() for _ in range(NL)]
    held_v = [dict() for _ in range(NL)]
    res = LoopResult(types=types, stats=stats)
    ev = lambda: torch.cuda.Event(enable_timing=True)
    for b in range(n_blocks):
        e0, e1 = ev(), ev()
        e0.record()
        cls_ms = 0.0
        for si, t in enumerate(steps):
            for layer in range(NL):
                q, k, v = block_data(layer, b, si)
                if tables_at_fill is not None and b == W - 1 and si == 0:
                    kw = torch.cat([held_k[layer][j] for j in range(b)] + [k], dim=1)
                    vw = torch.cat([held_v[layer][j] for j in range(b)] + [v], dim=1)
                    types[layer] = np.asarray(tables_at_fill[layer], np.uint8)
                    ctx.set_head_types(layer, types[layer], b, kw, vw)
                    del kw, vw
                elif classify and b == W - 1 and si == 0:
                    kw = torch.cat([held_k[layer][j] for j in range(b)] + [k], dim=1)
                    vw = torch.cat([held_v[layer][j] for j in range(b)] + [v], dim=1)
                    c0, c1 = ev(), ev()
                    c0.record()
                    types[layer], stats[layer] = ctx.classify_heads(layer, b, q, kw, vw)
                    c1.record()
                    c1.synchronize()
                    cls_ms += c0.elapsed_time(c1)
                    del kw, vw
                elif b == 0 and si == 0:
                    ctx.set_head_types(layer, types[layer], 0, k, v)
                else:
                    ctx.append_block(layer, b, k, v)
                if (classify or tables_at_fill is not None) and b < W - 1:
                    held_k[layer][b], held_v[layer][b] = k, v
                ctx.attention(layer, q, types[layer], out)
                if on_step is not None:
                    on_step(layer, b, si, types[layer], q)
        e1.record()
        e1.synchronize()
        res.ms_per_block.append(e0.elapsed_time(e1) - cls_ms)
        if cls_ms:
            res.classify_ms = cls_ms
            res.classified_at = b
        if b == W - 1:
            for layer in range(NL):          # the window is not needed any more
                held_k[layer].clear()
                held_v[layer].clear()
    return res
