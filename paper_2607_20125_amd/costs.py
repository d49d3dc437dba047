"""Algorithmic work of the routed-attention path, used to turn measured times
into TFLOP/s and GB/s.

FLOPs: the two matrix products of attention cost 4 * d flops per (query, key)
pair that is inside the query's key set (Appendix B counts 4 B Lq Lk d per
head); pairs outside the set -- masked work of the Spatial kernel -- are not
counted.  Compulsory bytes: what a head must move at least once: its bf16
queries, the bf16 K and V it attends to (its buffer's valid keys) and its fp32
output.
"""
from __future__ import annotations

SINK, DUMMY, SPATIAL, GLOBAL = 0, 1, 2, 3


def _window_extent_sum(n: int, r: int) -> int:
    """Sum over the n positions of one axis of the clipped window length."""
    return sum(min(i + r, n - 1) - max(i - r, 0) + 1 for i in range(n))


def pairs(kind: int, grid_h: int, grid_w: int, frames: int, n_blocks: int, r: int,
          sd_blocks: int = 1) -> int:
    L = frames * grid_h * grid_w
    if kind in (SINK, DUMMY):
        return L * min(sd_blocks, n_blocks) * L
    if kind == GLOBAL:
        return L * n_blocks * L
    return (frames * _window_extent_sum(grid_h, r) * _window_extent_sum(grid_w, r)
            * n_blocks * frames)


def cell_sizes(n: int, c: int) -> list:
    """Cell extents along one axis of the cell variant: round(n / c) cells,
    halves rounded up, c wide except the last, which ends at n."""
    k = max(1, (2 * n + c) // (2 * c))
    return [c] * (k - 1) + [n - c * (k - 1)]


def cell_pairs(grid_h: int, grid_w: int, frames: int, n_blocks: int, c: int) -> int:
    """In-set pairs of one Spatial head in the cell variant: each cell's
    frames * area queries against its n_blocks * frames * area keys."""
    return sum(frames * a * n_blocks * frames * a
               for a in (h * w for h in cell_sizes(grid_h, c) for w in cell_sizes(grid_w, c)))


def head_flops(kind, grid_h, grid_w, frames, n_blocks, r, d, cell=0, sd_blocks=1) -> int:
    if kind == SPATIAL and cell > 0:
        return 4 * d * cell_pairs(grid_h, grid_w, frames, n_blocks, cell)
    return 4 * d * pairs(kind, grid_h, grid_w, frames, n_blocks, r, sd_blocks)


def head_bytes(kind, grid_h, grid_w, frames, n_blocks, d) -> int:
    L = frames * grid_h * grid_w
    keys = L if kind in (SINK, DUMMY) else n_blocks * L
    return L * d * 2 + 2 * keys * d * 2 + L * d * 4


def layer_flops(types, grid_h, grid_w, frames, n_blocks, r, d, kinds=None, cell=0,
                sd_blocks=1) -> int:
    return sum(head_flops(int(t), grid_h, grid_w, frames, n_blocks, r, d, cell, sd_blocks)
               for t in types if kinds is None or int(t) in kinds)


def layer_bytes(types, grid_h, grid_w, frames, n_blocks, d, kinds=None) -> int:
    return sum(head_bytes(int(t), grid_h, grid_w, frames, n_blocks, d) for t in types
               if kinds is None or int(t) in kinds)


def append_bytes(n_heads, grid_h, grid_w, frames, d) -> int:
    """One block of K and V read and written once."""
    L = frames * grid_h * grid_w
    return 2 * 2 * n_heads * L * d * 2
