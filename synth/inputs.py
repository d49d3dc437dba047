"""Seeded synthetic inputs for HeadCast routed attention.

This module is shared by the tests, the benchmark and the CPU oracle's callers.
It only *draws* inputs: it holds none of the method's arithmetic (no attention,
no statistics, no decision rule, no cache layout).

Shapes follow the Wan-1.3B-class backbones the paper evaluates (30 layers x 12
heads, Appendix B / Table 6; 3 latent frames per block and a 7-block window,
Sec. 5.1) with head_dim 128 and the 480P / 720P / 1080P latent grids.
Values are i.i.d. N(0, 1) drawn in float32 and rounded to bfloat16 with
round-to-nearest-even; every tensor is returned as raw bf16 bit patterns
(uint16) so that both the GPU path and the oracle see identical bits.

Every (seed, layer, head, tensor, block) has its own numpy stream, so any
slice can be regenerated on its own.

Token order inside a block: t = f * (grid_h * grid_w) + y * grid_w + x.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

# archetype codes (same values as the C ABI's HC_SINK .. HC_GLOBAL)
SINK, DUMMY, SPATIAL, GLOBAL = 0, 1, 2, 3
TYPE_NAMES = ("sink", "dummy", "spatial", "global")

# tensor ids of the per-(layer, head, block) streams
T_Q, T_K, T_V, T_DIR, T_MIX = 0, 1, 2, 3, 4


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    n_layers: int
    n_heads: int
    head_dim: int
    grid_h: int
    grid_w: int
    frames_per_block: int
    window_blocks: int          # counts the current block
    spatial_radius: int         # deployed Spatial path radius r
    proxy_radius: int           # classification Spatial proxy radius r_p
    seed: int
    mix: tuple                  # head counts (sink, dummy, spatial, global) over all layers
    planted: bool = False       # classification workload with planted archetypes

    @property
    def tokens_per_frame(self) -> int:
        return self.grid_h * self.grid_w

    @property
    def block_tokens(self) -> int:          # L = Lq
        return self.frames_per_block * self.tokens_per_frame

    @property
    def window_tokens(self) -> int:         # Lk = W * L
        return self.window_blocks * self.block_tokens

    def scaled(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    # one head per archetype, fixed table (sink, dummy, spatial, global)
    "tiny": Workload("tiny", 1, 4, 64, 8, 8, 2, 4, 1, 2, 0, (1, 1, 1, 1)),
    "480p": Workload("480p", 30, 12, 128, 30, 52, 3, 7, 4, 2, 480, (90, 90, 90, 90)),
    "720p": Workload("720p", 30, 12, 128, 45, 80, 3, 7, 4, 2, 720, (72, 108, 108, 72)),
    "1080p": Workload("1080p", 30, 12, 128, 68, 120, 3, 7, 4, 2, 1080, (72, 108, 108, 72)),
    # classification + routing at 720P shapes with planted archetypes
    "classify720p": Workload("classify720p", 30, 12, 128, 45, 80, 3, 7, 4, 2, 1000,
                             (72, 108, 108, 72), planted=True),
    # the same recipe at the tiny shape (brute-force recovery of planted labels)
    "tiny_planted": Workload("tiny_planted", 1, 4, 64, 8, 8, 2, 4, 1, 2, 7,
                             (1, 1, 1, 1), planted=True),
}


def stream(seed: int, layer: int, head: int, tensor: int, block: int) -> np.random.Generator:
    return np.random.default_rng([seed, layer, head, tensor, block])


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit pattern, round to nearest even (finite inputs)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    # finite values stay below 0xFF800000, so the sum cannot wrap in 32 bits
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def head_types(w: Workload) -> np.ndarray:
    """Archetype table [n_layers][n_heads] (uint8).

    The tiny workload uses the fixed table (sink, dummy, spatial, global).
    Otherwise the exact multiset given by ``w.mix`` is shuffled with a seeded
    permutation and reshaped to [layers][heads].
    """
    if w.n_layers * w.n_heads == sum(w.mix) == 4 and w.n_heads == 4:
        return np.array([[SINK, DUMMY, SPATIAL, GLOBAL]], dtype=np.uint8)
    assert sum(w.mix) == w.n_layers * w.n_heads, (w.mix, w.n_layers, w.n_heads)
    flat = np.concatenate([np.full(c, t, dtype=np.uint8) for t, c in enumerate(w.mix)])
    perm = stream(w.seed, 0, 0, T_MIX, 0).permutation(flat.size)
    return flat[perm].reshape(w.n_layers, w.n_heads)


def _normal_bf16(w: Workload, layer: int, head: int, tensor: int, block: int) -> np.ndarray:
    g = stream(w.seed, layer, head, tensor, block)
    return g.standard_normal((w.block_tokens, w.head_dim), dtype=np.float32)


def _unit_direction(w: Workload, layer: int, head: int) -> np.ndarray:
    u = stream(w.seed, layer, head, T_DIR, 0).standard_normal(w.head_dim)
    return (u / np.linalg.norm(u)).astype(np.float32)


# ---------------------------------------------------------------------------
# Planted archetypes (classification workload)
#
#  * Sink heads:   Q = Z + sqrt(d) u,  K[block 0] += 3 u      (+3 logits on block 0)
#  * Dummy heads:  Q = Z + sqrt(d) u,  K[block >= c] += 3 u   (+3 logits on the current block c)
#  * Spatial heads: a logit term -0.5 * ((y - y')^2 + (x - x')^2) carried exactly
#    by the last N_COORD channels of Q and K (coordinates centred on the frame).
#  * Global heads: unbiased.
# u is a seeded unit vector per head; Z ~ N(0, 1).  With s = 1/sqrt(d), the
# +3 u shift lands as +3 (+- 0.27) logits because Q carries sqrt(d) u.
# ---------------------------------------------------------------------------
N_COORD = 7
SPATIAL_BETA = 1.0        # logit term is -SPATIAL_BETA/2 * squared distance
PLANT_SHIFT = 3.0


def _limbs(v: np.ndarray, n: int) -> list:
    """Split float64 values into n bf16 limbs whose sum approximates v."""
    out, rest = [], v.astype(np.float64)
    for _ in range(n):
        hi = bf16_bits_to_f32(f32_to_bf16_bits(rest.astype(np.float32))).astype(np.float64)
        out.append(hi)
        rest = rest - hi
    return out


def _coords(w: Workload):
    t = np.arange(w.block_tokens)
    pix = t % w.tokens_per_frame
    y = pix // w.grid_w - w.grid_h // 2
    x = pix % w.grid_w - w.grid_w // 2
    return y.astype(np.float64), x.astype(np.float64)


def _spatial_q_channels(w: Workload) -> np.ndarray:
    y, x = _coords(w)
    one = np.ones_like(y)
    return np.stack([y, y, x, x, one, one, one], axis=1)


def _spatial_k_channels(w: Workload) -> np.ndarray:
    y, x = _coords(w)
    a = math.sqrt(w.head_dim) * SPATIAL_BETA
    cy, cx = _limbs(a * y, 2), _limbs(a * x, 2)
    c2 = _limbs(-0.5 * a * (y * y + x * x), 3)
    return np.stack(cy + cx + c2, axis=1)


def gen_block(w: Workload, layer: int, head: int, tensor: int, block: int,
              classify_block: int | None = None) -> np.ndarray:
    """One block of Q, K or V for one head: bf16 bits [L][d].

    ``tensor`` is T_Q, T_K or T_V.  For planted workloads ``classify_block``
    (the block at which classification runs) selects the Dummy shift.
    """
    z = _normal_bf16(w, layer, head, tensor, block)
    if w.planted:
        kind = int(head_types(w)[layer, head])
        d = w.head_dim
        if kind in (SINK, DUMMY):
            u = _unit_direction(w, layer, head)
            if tensor == T_Q:
                z = z + np.float32(math.sqrt(d)) * u
            elif tensor == T_K:
                c = w.window_blocks - 1 if classify_block is None else classify_block
                if (kind == SINK and block == 0) or (kind == DUMMY and block >= c):
                    z = z + np.float32(PLANT_SHIFT) * u
        elif kind == SPATIAL and tensor in (T_Q, T_K):
            ch = _spatial_q_channels(w) if tensor == T_Q else _spatial_k_channels(w)
            z = z.copy()
            z[:, d - N_COORD:] = ch.astype(np.float32)
    return f32_to_bf16_bits(z)


def window_block_ids(cur_block: int, window_blocks: int) -> list:
    """Block ids held by the window at ``cur_block``, in the order the ABI
    expects them: the sink block 0 first, then the most recent blocks, oldest
    first, ending with the current block (input contract of k_win / v_win)."""
    if cur_block < window_blocks - 1:
        return list(range(cur_block + 1))
    return [0] + list(range(cur_block - window_blocks + 2, cur_block + 1))


def gen_layer(w: Workload, layer: int, cur_block: int, heads=None,
              classify_block: int | None = None):
    """Q [H][L][d], K_win and V_win [H][n*L][d] (bf16 bits) for one layer."""
    heads = range(w.n_heads) if heads is None else heads
    ids = window_block_ids(cur_block, w.window_blocks)
    q = np.stack([gen_block(w, layer, h, T_Q, cur_block, classify_block) for h in heads])
    k = np.stack([np.concatenate([gen_block(w, layer, h, T_K, b, classify_block) for b in ids])
                  for h in heads])
    v = np.stack([np.concatenate([gen_block(w, layer, h, T_V, b, classify_block) for b in ids])
                  for h in heads])
    return q, k, v


def gen_step_block(w: Workload, layer: int, block: int, heads=None,
                   classify_block: int | None = None):
    """Q, K, V of one block for all heads [H][L][d] (bf16 bits)."""
    heads = range(w.n_heads) if heads is None else heads
    q = np.stack([gen_block(w, layer, h, T_Q, block, classify_block) for h in heads])
    k = np.stack([gen_block(w, layer, h, T_K, block, classify_block) for h in heads])
    v = np.stack([gen_block(w, layer, h, T_V, block, classify_block) for h in heads])
    return q, k, v


def device_normal_bf16(shape, seed: int, device):
    """Large benchmark inputs drawn on the device: N(0,1) float32 rounded to
    bf16 (torch's conversion is round-to-nearest-even)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return torch.randn(shape, generator=g, device=device, dtype=torch.float32).to(torch.bfloat16)
