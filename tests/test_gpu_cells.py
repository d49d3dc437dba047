"""GPU parity of the cell variant of the Spatial path (Sec. 4.4; 10 x 10 cells in
Sec. 5.1): every query attends to its own c x c cell in every window frame.
The HIP path (C ABI, `spatial_cell` = c) against the oracle's cell key sets on
the same seeded bf16 inputs; max-abs 1e-2, mean-abs 1e-3."""
import numpy as np
import pytest

from helpers import assert_close, dev_bf16, out_tensor, stratified_rows
from oracle import headcast_oracle as O
from synth import inputs as S

pytestmark = pytest.mark.gpu


def oracle_cells(w, types, q, k, v, c, rows=None):
    return O.routed_attention(types, q, k, v, w.grid_h, w.grid_w, w.frames_per_block,
                              w.spatial_radius, rows=rows, spatial_cell=c)


def gpu_cells(hc, w, types, cur, q, k, v, c):
    import torch
    ctx = hc.Context(hc.config_from_workload(w, n_layers=1, spatial_cell=c), 0)
    ctx.set_head_types(0, types, cur, dev_bf16(k), dev_bf16(v))
    o = out_tensor(w)
    ctx.attention(0, dev_bf16(q), types, o)
    torch.cuda.synchronize()
    return ctx, o.cpu().numpy()


@pytest.mark.parametrize("cur", [0, 1, 3, 6])
def test_tiny_fixed_table_cells(hc, cur):
    w = S.WORKLOADS["tiny"]
    types = S.head_types(w)[0]
    q, k, v = S.gen_layer(w, 0, cur)
    _, got = gpu_cells(hc, w, types, cur, q, k, v, 3)
    assert_close(got, oracle_cells(w, types, q, k, v, 3), f"tiny cells c=3 cur={cur}")


@pytest.mark.parametrize("c", [2, 3, 5, 8])
def test_tiny_all_spatial_cell_sizes(hc, c):
    w = S.WORKLOADS["tiny"]
    types = np.full(w.n_heads, S.SPATIAL, np.uint8)
    cur = w.window_blocks - 1
    q, k, v = S.gen_layer(w, 0, cur, heads=range(w.n_heads))
    _, got = gpu_cells(hc, w, types, cur, q, k, v, c)
    assert_close(got, oracle_cells(w, types, q, k, v, c), f"tiny all-Spatial c={c}")
    if c == 8:      # one cell covers the frame: the Global path
        glob = O.routed_attention(np.full(w.n_heads, S.GLOBAL, np.uint8), q, k, v, w.grid_h,
                                  w.grid_w, w.frames_per_block, w.spatial_radius)
        assert_close(got, glob, "one cell vs Global")


def test_ragged_grid_cells(hc):
    # 5 x 8 frame (cells 5/2 -> 3 rows of 2, 2, 1; 8/2 -> 4), head_dim 128
    w = S.Workload("ragged", 1, 6, 128, 5, 8, 1, 3, 2, 2, 11, (1, 2, 2, 1))
    types = np.array([3, 2, 0, 1, 2, 3], np.uint8)
    for cur in (1, 2, 4):
        q, k, v = S.gen_layer(w, 0, cur)
        _, got = gpu_cells(hc, w, types, cur, q, k, v, 2)
        assert_close(got, oracle_cells(w, types, q, k, v, 2), f"ragged cells cur={cur}")


def test_tiny_cells_across_appends(hc):
    import torch
    w = S.WORKLOADS["tiny"]
    types = np.array([2, 3, 2, 1], np.uint8)
    ctx = hc.Context(hc.config_from_workload(w, spatial_cell=3), 0)
    q, k, v = S.gen_layer(w, 0, 0)
    ctx.set_head_types(0, types, 0, dev_bf16(k), dev_bf16(v))
    for b in range(1, 3 * w.window_blocks):
        qb, kb, vb = S.gen_step_block(w, 0, b)
        ctx.append_block(0, b, dev_bf16(kb), dev_bf16(vb))
        o = out_tensor(w)
        ctx.attention(0, dev_bf16(qb), types, o)
        torch.cuda.synchronize()
        _, kw, vw = S.gen_layer(w, 0, b)
        assert_close(o.cpu().numpy(), oracle_cells(w, types, qb, kw, vw, 3), f"cells b={b}")


def test_480p_full_layer_cells(hc):
    w = S.WORKLOADS["480p"]
    types = S.head_types(w)[0]
    cur = w.window_blocks - 1
    print("480p layer 0 generate", flush=True)
    q, k, v = S.gen_layer(w, 0, cur)
    print("480p cells gpu", flush=True)
    _, got = gpu_cells(hc, w, types, cur, q, k, v, 10)
    print("480p cells oracle", flush=True)
    assert_close(got, oracle_cells(w, types, q, k, v, 10), "480p cells c=10")


@pytest.mark.parametrize("name", ["720p", "1080p"])
def test_sampled_rows_cells(hc, name):
    w = S.WORKLOADS[name]
    layer = 2
    types = S.head_types(w)[layer]
    cur = w.window_blocks - 1
    print(f"{name} layer {layer} generate", flush=True)
    q, k, v = S.gen_layer(w, layer, cur)
    _, got = gpu_cells(hc, w, types, cur, q, k, v, 10)
    rows = stratified_rows(w, n_random=256, seed=3)
    print(f"{name} cells oracle on {rows.size} rows", flush=True)
    assert_close(got[:, rows], oracle_cells(w, types, q, k, v, 10, rows=rows), f"{name} cells")
