"""HeadCast routed attention: plain CPU oracle (float64).

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module.  It shares no code
with the GPU library (no kernels, headers, helpers or tables); both sides only
share the seeded input generator in ``synth/``.

Everything here is the plain definition written out, in float64:

* attention of a query over an explicit key set S:
      o = sum_{k in S} exp(s q.k - m) v_k / sum_{k in S} exp(s q.k - m),
      m = max_{k in S} s q.k,  s = 1/sqrt(d) unless configured otherwise;
* the four archetype key sets (Sec. 4.2 proxies, Sec. 4.4 paths);
* the classification statistics and decision rule (Sec. 4.2, Eq. 3-5);
* the cache-layout integers (Sec. 4.3): ring slots and per-buffer head slots.

Readings of points the paper leaves open:
  R1 Sink = the L keys of block 0; Dummy = the L keys of the current block
     (the proxies of Sec. 4.2; each path of Sec. 4.4 attends to a single block).
  R2 Spatial = all frames of the window (current block included), restricted
     to |y'-y| <= r and |x'-x| <= r, clipped at the frame border.
  R3 the window W counts the current block; block 0 is the frozen sink block.
  R4 cos with a zero vector uses max(|a||b|, 1e-30) as the denominator.
  R5 P5 = linear interpolation at rank 0.05 (n-1) of the ascending values.
  R6 MSE = mean over all L_q * d elements of the raw outputs.
  R7 Eq. 5 comparisons are inclusive, in the order Sink, Dummy, Spatial, Global.
  R1 alt (sd_blocks = 2): Sink = block 0 + the current block, Dummy = the
     previous + the current block (App. B / App. C cost them at 2L).
  R20 cell variant of the Spatial path: round(N / c) cells per axis (halves
     rounded up, at least one), c positions each, the last cell ending at N.

Parity status: every function below is pinned by ``tests/test_oracle_pins.py``
(closed forms, invariants, library routines, brute force); none is unpinned.

Inputs are bf16 bit patterns (uint16) widened exactly to float64.
"""
from __future__ import annotations

import math

import numpy as np
import torch

SINK, DUMMY, SPATIAL, GLOBAL = 0, 1, 2, 3

# Sec. 5.1 (implementation details): thresholds, MSE weight, proxy radius.
THETA = 0.95          # theta_s = theta_d = theta_sp
THETA_SCORE = 0.755   # theta_sc
GAMMA = 5.0           # gamma in Eq. 4
COS_EPS = 1e-30


def widen(bits) -> np.ndarray:
    """bf16 bit patterns -> float64 (exact)."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _t(x) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float64))


# ---------------------------------------------------------------------------
# Window and cache layout (Sec. 3.1 sliding window with a fixed sink block;
# Sec. 4.3 heterogeneous cache management)
# ---------------------------------------------------------------------------
def window_blocks(cur_block: int, W: int) -> list:
    """Blocks visible at ``cur_block``: the frozen sink block 0 plus the most
    recent blocks, W in total counting the current one (reading R3)."""
    if cur_block < W - 1:
        return list(range(cur_block + 1))
    return [0] + list(range(cur_block - W + 2, cur_block + 1))


def simulate_ring(blocks_seen: int, W: int) -> dict:
    """Physical slot of every block still cached after blocks 0..blocks_seen-1
    were written, simulated step by step: slot 0 holds block 0 forever; every
    later block takes an empty slot if one is left, else the slot of the oldest
    rolling block (the one the sliding window evicts)."""
    slot_of = {}
    for b in range(blocks_seen):
        if b == 0:
            slot_of[0] = 0
            continue
        used = set(slot_of.values())
        free = [s for s in range(1, W) if s not in used]
        if free:
            slot_of[b] = free[0]
        else:
            oldest = min(k for k in slot_of if k != 0)
            slot_of[b] = slot_of.pop(oldest)
    return slot_of


def ring_slots_of_logical(cur_block: int, W: int) -> list:
    """Physical slot of each logical window position (sink first, current
    last); -1 where the window is not yet full."""
    held = simulate_ring(cur_block + 1, W)
    ids = window_blocks(cur_block, W)
    out = [held[b] for b in ids]
    return out + [-1] * (W - len(out))


def head_slots(types) -> list:
    """Index of each head inside its buffer (Sec. 4.3): Sink and Dummy heads
    share the Sink-Dummy buffer, Global and Spatial heads have their own;
    heads keep their head-id order inside a buffer."""
    buf = {SINK: 0, DUMMY: 0, SPATIAL: 2, GLOBAL: 3}
    count = {0: 0, 2: 0, 3: 0}
    out = []
    for t in types:
        b = buf[int(t)]
        out.append(count[b])
        count[b] += 1
    return out


# ---------------------------------------------------------------------------
# Key sets (Sec. 4.2 proxies; Sec. 4.4 paths)
# Keys are indexed in logical window order: key j is token j % L of logical
# block j // L; token t = f*Hg*Wg + y*Wg + x.
# ---------------------------------------------------------------------------
class Geometry:
    def __init__(self, grid_h, grid_w, frames_per_block, n_blocks):
        self.Hg, self.Wg, self.F, self.n = grid_h, grid_w, frames_per_block, n_blocks
        self.P = grid_h * grid_w
        self.L = frames_per_block * self.P

    def yx(self, t):
        p = t % self.P
        return p // self.Wg, p % self.Wg


def keys_global(g: Geometry, t: int) -> np.ndarray:
    return np.arange(g.n * g.L)


def keys_sink(g: Geometry, t: int, blocks: int = 1) -> np.ndarray:
    """Logical block 0; with blocks = 2 also the current block (App. B / C:
    anchor + current)."""
    if blocks == 2 and g.n >= 2:
        return np.concatenate([np.arange(g.L), np.arange((g.n - 1) * g.L, g.n * g.L)])
    return np.arange(g.L)


def keys_dummy(g: Geometry, t: int, blocks: int = 1) -> np.ndarray:
    """The current block; with blocks = 2 also the previous one (App. B / C:
    previous + current)."""
    first = g.n - 2 if (blocks == 2 and g.n >= 2) else g.n - 1
    return np.arange(first * g.L, g.n * g.L)


def keys_spatial(g: Geometry, t: int, r: int) -> np.ndarray:
    """All window frames, positions with |y'-y| <= r and |x'-x| <= r inside
    the frame (readings R2, clipped square window)."""
    y, x = g.yx(t)
    ys = np.arange(max(0, y - r), min(g.Hg - 1, y + r) + 1)
    xs = np.arange(max(0, x - r), min(g.Wg - 1, x + r) + 1)
    pix = (ys[:, None] * g.Wg + xs[None, :]).ravel()
    frames = np.arange(g.n * g.F)
    return (frames[:, None] * g.P + pix[None, :]).ravel()


def cell_bounds(N: int, c: int) -> np.ndarray:
    """Cell boundaries along one axis of the deployed Spatial path (Sec. 4.4
    and Sec. 5.1: non-overlapping c x c cells, the boundary remainder rounded):
    round(N / c) cells, halves rounded up, at least one; every cell has c
    positions except the last, which ends at N (reading R20)."""
    n = max(1, int(math.floor(N / c + 0.5)))
    return np.array([i * c for i in range(n)] + [N])


def keys_spatial_cell(g: Geometry, t: int, c: int) -> np.ndarray:
    """All window frames, positions inside the c x c cell that holds the
    query's position (Sec. 4.4 Spatial path, cell variant)."""
    y, x = g.yx(t)
    by, bx = cell_bounds(g.Hg, c), cell_bounds(g.Wg, c)
    cy = int(np.searchsorted(by, y, side="right")) - 1
    cx = int(np.searchsorted(bx, x, side="right")) - 1
    ys = np.arange(by[cy], by[cy + 1])
    xs = np.arange(bx[cx], bx[cx + 1])
    pix = (ys[:, None] * g.Wg + xs[None, :]).ravel()
    frames = np.arange(g.n * g.F)
    return (frames[:, None] * g.P + pix[None, :]).ravel()


def key_set(kind: int, g: Geometry, t: int, r: int, sd_blocks: int = 1) -> np.ndarray:
    if kind == SINK:
        return keys_sink(g, t, sd_blocks)
    if kind == DUMMY:
        return keys_dummy(g, t, sd_blocks)
    if kind == SPATIAL:
        return keys_spatial(g, t, r)
    return keys_global(g, t)


# ---------------------------------------------------------------------------
# Softmax attention over explicit key sets
# ---------------------------------------------------------------------------
def attend_one(q, K, V, idx, scale) -> np.ndarray:
    """Plain definition for one query (pure numpy, small cases)."""
    logits = scale * (K[idx] @ q)
    m = logits.max()
    w = np.exp(logits - m)
    return (w[:, None] * V[idx]).sum(0) / w.sum()


def attend_shared(Q, K, V, scale, chunk=1024) -> np.ndarray:
    """Every row of Q attends to every row of K/V (all queries share one key
    set).  Query rows are independent, so they are processed in chunks."""
    Kt, Vt = _t(K), _t(V)
    out = np.empty((Q.shape[0], V.shape[1]))
    for a in range(0, Q.shape[0], chunk):
        s = scale * (_t(Q[a:a + chunk]) @ Kt.T)
        s = s - s.max(dim=1, keepdim=True).values
        w = torch.exp(s)
        out[a:a + chunk] = ((w @ Vt) / w.sum(dim=1, keepdim=True)).numpy()
    return out


def attend_spatial(Q, K, V, g: Geometry, r: int, scale, rows=None, batch=64) -> np.ndarray:
    """Spatial key sets: query t sees keys_spatial(g, t, r).  Queries at the
    same (y, x) share that set, so they are grouped by position; within a batch
    of positions the explicit index lists are padded to a common length and
    the padding is excluded from the softmax (weight exactly zero)."""
    rows = np.arange(Q.shape[0]) if rows is None else np.asarray(rows)
    out = np.empty((rows.size, V.shape[1]))
    pos = rows % g.P
    uniq = np.unique(pos)
    Kt, Vt = _t(K), _t(V)
    for a in range(0, uniq.size, batch):
        ps = uniq[a:a + batch]
        sets = [keys_spatial(g, int(p), r) for p in ps]
        n = max(s.size for s in sets)
        idx = np.zeros((ps.size, n), dtype=np.int64)
        valid = np.zeros((ps.size, n), dtype=bool)
        for i, s in enumerate(sets):
            idx[i, :s.size] = s
            valid[i, :s.size] = True
        Kg = Kt[torch.from_numpy(idx)]          # [P, n, d]
        Vg = Vt[torch.from_numpy(idx)]
        for i, p in enumerate(ps):
            sel = np.nonzero(pos == p)[0]
            s = scale * (_t(Q[rows[sel]]) @ Kg[i].T)            # [nq, n]
            s = s.masked_fill(~torch.from_numpy(valid[i])[None, :], -math.inf)
            s = s - s.max(dim=1, keepdim=True).values
            w = torch.exp(s)
            out[sel] = ((w @ Vg[i]) / w.sum(dim=1, keepdim=True)).numpy()
    return out


def attend_cells(Q, K, V, g: Geometry, c: int, scale, rows=None) -> np.ndarray:
    """Cell variant of the Spatial path: every query of a cell shares the
    cell's key set, so each cell is one dense attention."""
    rows = np.arange(Q.shape[0]) if rows is None else np.asarray(rows)
    out = np.empty((rows.size, V.shape[1]))
    by, bx = cell_bounds(g.Hg, c), cell_bounds(g.Wg, c)
    ys, xs = g.yx(rows)
    cy = np.searchsorted(by, ys, side="right") - 1
    cx = np.searchsorted(bx, xs, side="right") - 1
    cell = cy * (bx.size - 1) + cx
    for cid in np.unique(cell):
        sel = np.nonzero(cell == cid)[0]
        ks = keys_spatial_cell(g, int(rows[sel[0]]), c)
        out[sel] = attend_shared(Q[rows[sel]], K[ks], V[ks], scale)
    return out


def attend_kind(kind, Q, K, V, g: Geometry, r, scale, rows=None, cell=0,
                sd_blocks=1) -> np.ndarray:
    """Output of one head of archetype ``kind`` for query rows ``rows`` of the
    current block (all rows when None).  Q: [L][d]; K, V: [n*L][d] (logical
    window order), float64.  Spatial heads use the centred (2r+1)^2 window, or
    c x c cells when ``cell`` = c > 0; Sink and Dummy heads one block, or two
    when ``sd_blocks`` = 2."""
    rows = np.arange(Q.shape[0]) if rows is None else np.asarray(rows)
    if kind == SPATIAL:
        if cell > 0:
            return attend_cells(Q, K, V, g, cell, scale, rows)
        return attend_spatial(Q, K, V, g, r, scale, rows)
    t0 = int(rows[0]) if rows.size else 0
    ks = key_set(kind, g, t0, r, sd_blocks)    # the same set for every query
    return attend_shared(Q[rows], K[ks], V[ks], scale)


def routed_attention(types, q_bits, k_bits, v_bits, grid_h, grid_w, frames_per_block,
                     spatial_radius, scale=None, rows=None, spatial_cell=0,
                     sd_blocks=1) -> np.ndarray:
    """Sec. 4.4: every head attends over the key set of its archetype.
    q_bits [H][L][d]; k_bits, v_bits [H][n*L][d] in logical window order.
    ``spatial_cell`` > 0 selects the cell variant of the Spatial path,
    ``sd_blocks`` = 2 the two-block Sink / Dummy variant (reading R1 alt).
    Returns float64 [H][len(rows)][d]."""
    H, L, d = q_bits.shape
    n = k_bits.shape[1] // L
    g = Geometry(grid_h, grid_w, frames_per_block, n)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    return np.stack([attend_kind(int(types[h]), widen(q_bits[h]), widen(k_bits[h]),
                                 widen(v_bits[h]), g, spatial_radius, scale, rows,
                                 spatial_cell, sd_blocks)
                     for h in range(H)])


# ---------------------------------------------------------------------------
# Online classification (Sec. 4.2, Eq. 2-5)
# ---------------------------------------------------------------------------
def token_cos(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """cos(a[t], b[t]) for every token t (reading R4 for zero vectors)."""
    num = (a * b).sum(1)
    den = np.sqrt((a * a).sum(1)) * np.sqrt((b * b).sum(1))
    return num / np.maximum(den, COS_EPS)


def percentile5(x: np.ndarray) -> float:
    """5th percentile by linear interpolation between the ascending order
    statistics at rank 0.05 (n - 1) (reading R5)."""
    s = np.sort(np.asarray(x, dtype=np.float64))
    rank = 0.05 * (s.size - 1)
    lo = int(math.floor(rank))
    hi = min(lo + 1, s.size - 1)
    return float(s[lo] + (rank - lo) * (s[hi] - s[lo]))


def head_statistics(o_ref, o_sink, o_dummy, o_sp, gamma=GAMMA) -> np.ndarray:
    """[cos_sink, cos_dummy, cos_spatial, P5(cos_spatial), MSE, score] of one
    head (Eq. 3 and Eq. 4)."""
    c_sink = token_cos(o_sink, o_ref)
    c_dummy = token_cos(o_dummy, o_ref)
    c_sp = token_cos(o_sp, o_ref)
    p5 = percentile5(c_sp)
    mse = float(((o_sp - o_ref) ** 2).mean())
    return np.array([c_sink.mean(), c_dummy.mean(), c_sp.mean(), p5, mse, p5 - gamma * mse])


def decide(stats, theta_s=THETA, theta_d=THETA, theta_sp=THETA, theta_sc=THETA_SCORE) -> int:
    """Mutually exclusive decision hierarchy (Eq. 5)."""
    cos_sink, cos_dummy, cos_sp, _p5, _mse, score = stats
    if cos_sink >= theta_s:
        return SINK
    if cos_dummy >= theta_d:
        return DUMMY
    if cos_sp >= theta_sp and score >= theta_sc:
        return SPATIAL
    return GLOBAL


def proxy_outputs(q, k, v, g: Geometry, proxy_radius, scale):
    """O_ref (Eq. 2) and the three restricted outputs of one head: Sink proxy
    (first block), Dummy proxy (current block), Spatial proxy (all window frames,
    (2 r_p + 1)^2 grid around the query)."""
    return (attend_kind(GLOBAL, q, k, v, g, proxy_radius, scale),
            attend_kind(SINK, q, k, v, g, proxy_radius, scale),
            attend_kind(DUMMY, q, k, v, g, proxy_radius, scale),
            attend_kind(SPATIAL, q, k, v, g, proxy_radius, scale))


def classify_layer(q_bits, k_bits, v_bits, grid_h, grid_w, frames_per_block, proxy_radius,
                   scale=None, gamma=GAMMA, theta=THETA, theta_sc=THETA_SCORE):
    """Labels [H] (uint8) and statistics [H][6] for one layer."""
    H, L, d = q_bits.shape
    n = k_bits.shape[1] // L
    g = Geometry(grid_h, grid_w, frames_per_block, n)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    labels, stats = [], []
    for h in range(H):
        outs = proxy_outputs(widen(q_bits[h]), widen(k_bits[h]), widen(v_bits[h]),
                             g, proxy_radius, scale)
        st = head_statistics(*outs, gamma=gamma)
        stats.append(st)
        labels.append(decide(st, theta, theta, theta, theta_sc))
    return np.array(labels, dtype=np.uint8), np.stack(stats)


# ---------------------------------------------------------------------------
# Cost models
# ---------------------------------------------------------------------------
def in_set_pairs(kind, grid_h, grid_w, frames_per_block, n_blocks, r) -> int:
    """Number of (query, key) pairs of one head: the sum over the current
    block's queries of the size of their key set."""
    g = Geometry(grid_h, grid_w, frames_per_block, n_blocks)
    if kind in (SINK, DUMMY):
        return g.L * g.L
    if kind == GLOBAL:
        return g.L * g.n * g.L

    def count(N):   # sum over positions of the clipped window extent
        i = np.arange(N)
        return int((np.minimum(i + r, N - 1) - np.maximum(i - r, 0) + 1).sum())
    return g.F * count(grid_h) * count(grid_w) * g.n * g.F


def algorithmic_flops(types, grid_h, grid_w, frames_per_block, n_blocks, r, d) -> int:
    """4 d flops per in-set (query, key) pair (QK^T and PV, Appendix B)."""
    return sum(4 * d * in_set_pairs(int(t), grid_h, grid_w, frames_per_block, n_blocks, r)
               for t in types)


def paper_flop_ratio(n_s, n_d, n_sp, n_g, n_total=None) -> float:
    """Appendix B: (2 N_s + 2 N_d + N_sp / 2 + 8 N_g) / (8 N_total).  N_total is
    the number of heads (the per-type counts of Table 6 are rounded means)."""
    n = n_s + n_d + n_sp + n_g if n_total is None else n_total
    return (2 * n_s + 2 * n_d + 0.5 * n_sp + 8 * n_g) / (8 * n)


def paper_kv_reduction(n_sd_fraction) -> float:
    """Appendix C: steady-state KV reduction (N_s + N_d) / N_total * 0.75."""
    return n_sd_fraction * 0.75
