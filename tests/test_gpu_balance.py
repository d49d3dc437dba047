"""GPU parity of dense launches whose unit lists are tail-balanced: with few
units per XCD the host cuts the last round's units into pieces of whole key
tiles (partial slots merged by the combine kernel), including Sink/Dummy units
that otherwise write their output directly.  480P-shaped layers with 2-4 heads
(296, 518 and 814 units: all of them are cut on a 256-CU MI355X), full tensors
against the oracle; max-abs 1e-2, mean-abs 1e-3."""
import numpy as np
import pytest

from helpers import assert_close, dev_bf16, out_tensor
from oracle import headcast_oracle as O
from synth import inputs as S

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("types", [(0, 3), (3, 3), (1, 3, 3, 3)])
def test_balanced_tail_480p(hc, types):
    import torch
    types = np.array(types, np.uint8)
    w = S.Workload("bal", 1, len(types), 128, 30, 52, 3, 7, 4, 2, 481, (0, 0, 0, len(types)))
    cur = w.window_blocks - 1
    print(f"balanced tail types={types.tolist()} generate", flush=True)
    q, k, v = S.gen_layer(w, 0, cur)
    ctx = hc.Context(hc.config_from_workload(w), 0)
    ctx.set_head_types(0, types, cur, dev_bf16(k), dev_bf16(v))
    o = out_tensor(w)
    ctx.attention(0, dev_bf16(q), types, o)
    torch.cuda.synchronize()
    print("oracle", flush=True)
    ref = O.routed_attention(types, q, k, v, w.grid_h, w.grid_w, w.frames_per_block,
                             w.spatial_radius)
    assert_close(o.cpu().numpy(), ref, f"balanced tail types={types.tolist()}")
