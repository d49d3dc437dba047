"""GPU parity over seeded random small configurations: grid shape, frames per
block, window length, Spatial radius, head dimension, head count and table,
window fill level, the cell variant and the two-block Sink/Dummy variant drawn
at random (only shapes the ABI accepts), each layer checked against the oracle
on every query.  Tolerance as elsewhere: max-abs 1e-2, mean-abs 1e-3."""
import numpy as np
import pytest

from helpers import assert_close, dev_bf16, out_tensor
from oracle import headcast_oracle as O
from synth import inputs as S

pytestmark = pytest.mark.gpu

N_CASES = 24


def draw(i):
    rng = np.random.default_rng([2607, i])
    while True:
        hg, wg = int(rng.integers(1, 13)), int(rng.integers(1, 17))
        f = int(rng.integers(1, 5))
        if (hg * wg * f) % 8 == 0 and hg * wg * f <= 640:
            break
    W = int(rng.integers(2, 7))
    r = int(rng.integers(0, 6))
    d = int(rng.choice([64, 128]))
    H = int(rng.integers(1, 9))
    types = rng.integers(0, 4, size=H).astype(np.uint8)
    cur = int(rng.integers(0, 3 * W))
    cell = int(rng.choice([0, 0, 2, 3, 5]))
    sd = int(rng.choice([1, 1, 2]))
    if W < 3:          # the two-block Dummy set needs the previous block in the window
        sd = 1
    return hg, wg, f, W, r, d, H, types, cur, cell, sd


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_config(hc, i):
    import torch
    hg, wg, f, W, r, d, H, types, cur, cell, sd = draw(i)
    w = S.Workload(f"rand{i}", 1, H, d, hg, wg, f, W, r, 2, 9000 + i, (H, 0, 0, 0))
    print(f"case {i}: grid {hg}x{wg} F={f} W={W} r={r} d={d} H={H} types={types.tolist()} "
          f"cur={cur} cell={cell} sd_blocks={sd}", flush=True)
    q, k, v = S.gen_layer(w, 0, cur)
    cfg = hc.config_from_workload(w, spatial_cell=cell, sd_blocks=sd)
    assert hc.validate_config(cfg) == hc.HC_OK
    ctx = hc.Context(cfg, 0)
    if sd == 2 and cur > 0:
        # the two-block variant needs the previous block: fill the window block by block
        for b in range(cur + 1):
            _, kb, vb = S.gen_step_block(w, 0, b)
            if b == 0:
                ctx.set_head_types(0, types, 0, dev_bf16(kb), dev_bf16(vb))
            else:
                ctx.append_block(0, b, dev_bf16(kb), dev_bf16(vb))
    else:
        ctx.set_head_types(0, types, cur, dev_bf16(k), dev_bf16(v))
    o = out_tensor(w)
    ctx.attention(0, dev_bf16(q), types, o)
    torch.cuda.synchronize()
    ref = O.routed_attention(types, q, k, v, hg, wg, f, r, spatial_cell=cell, sd_blocks=sd)
    assert_close(o.cpu().numpy(), ref, f"case {i}")
