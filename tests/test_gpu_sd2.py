"""GPU parity of the two-block Sink / Dummy variant (`sd_blocks` = 2; App. B and
App. C cost these heads at 2L): Sink attends to block 0 and the current block,
Dummy to the previous and the current block.  The HIP path (C ABI) against the
oracle's key sets on the same seeded bf16 inputs; max-abs 1e-2, mean-abs 1e-3."""
import numpy as np
import pytest

from helpers import assert_close, dev_bf16, out_tensor, stratified_rows
from oracle import headcast_oracle as O
from synth import inputs as S

pytestmark = pytest.mark.gpu


def oracle_sd2(w, types, q, k, v, rows=None):
    return O.routed_attention(types, q, k, v, w.grid_h, w.grid_w, w.frames_per_block,
                              w.spatial_radius, rows=rows, sd_blocks=2)


def gpu_sd2(hc, w, types, cur, q, k, v):
    import torch
    ctx = hc.Context(hc.config_from_workload(w, n_layers=1, sd_blocks=2), 0)
    ctx.set_head_types(0, types, cur, dev_bf16(k), dev_bf16(v))
    o = out_tensor(w)
    ctx.attention(0, dev_bf16(q), types, o)
    torch.cuda.synchronize()
    return o.cpu().numpy()


@pytest.mark.parametrize("cur", [0, 1, 2, 3, 6])
def test_tiny_fixed_table_two_blocks(hc, cur):
    w = S.WORKLOADS["tiny"]
    types = S.head_types(w)[0]
    q, k, v = S.gen_layer(w, 0, cur)
    got = gpu_sd2(hc, w, types, cur, q, k, v)
    assert_close(got, oracle_sd2(w, types, q, k, v), f"tiny sd2 cur={cur}")


def test_tiny_two_blocks_across_appends_with_overwrite(hc):
    import torch
    w = S.WORKLOADS["tiny"]
    types = np.array([0, 1, 1, 0], np.uint8)
    ctx = hc.Context(hc.config_from_workload(w, sd_blocks=2), 0)
    q, k, v = S.gen_layer(w, 0, 0)
    ctx.set_head_types(0, types, 0, dev_bf16(k), dev_bf16(v))
    other = w.scaled(seed=77)
    for b in range(1, 3 * w.window_blocks):
        _, kb0, vb0 = S.gen_step_block(other, 0, b)       # stale write, then the real one
        ctx.append_block(0, b, dev_bf16(kb0), dev_bf16(vb0))
        qb, kb, vb = S.gen_step_block(w, 0, b)
        ctx.append_block(0, b, dev_bf16(kb), dev_bf16(vb))
        o = out_tensor(w)
        ctx.attention(0, dev_bf16(qb), types, o)
        torch.cuda.synchronize()
        _, kw, vw = S.gen_layer(w, 0, b)
        assert_close(o.cpu().numpy(), oracle_sd2(w, types, qb, kw, vw), f"sd2 b={b}")


def test_480p_full_layer_two_blocks(hc):
    w = S.WORKLOADS["480p"]
    types = S.head_types(w)[1]
    cur = w.window_blocks - 1
    q, k, v = S.gen_layer(w, 1, cur)
    got = gpu_sd2(hc, w, types, cur, q, k, v)
    assert_close(got, oracle_sd2(w, types, q, k, v), "480p sd2")


def test_720p_sampled_two_blocks(hc):
    w = S.WORKLOADS["720p"]
    types = S.head_types(w)[4]
    cur = w.window_blocks - 1
    q, k, v = S.gen_layer(w, 4, cur)
    got = gpu_sd2(hc, w, types, cur, q, k, v)
    rows = stratified_rows(w, n_random=256, seed=4)
    assert_close(got[:, rows], oracle_sd2(w, types, q, k, v, rows=rows), "720p sd2")
