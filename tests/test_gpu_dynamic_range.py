"""GPU parity at logit magnitudes far from unit variance.  The dense and Spatial
kernels first run a pass with the softmax offset fixed at 0 and fall back to the
running-max pass when a row sum leaves [2^-60, 2^96] (overflow or underflow of
2^x); these inputs drive both branches, the merge of per-block Global partials
and of split Spatial partials produced by different passes.  The oracle is the
plain fp64 definition (max subtracted), so any magnitude is exact there.
Tolerance as elsewhere: max-abs 1e-2, mean-abs 1e-3."""
import numpy as np
import pytest

from helpers import assert_close, dev_bf16, out_tensor
from oracle import headcast_oracle as O
from synth import inputs as S

pytestmark = pytest.mark.gpu

# d = 128, 12 x 16 grid, 2 frames per block (L = 384, three 128-query tiles),
# window of 3 blocks (1152 keys), r = 1
W_RANGE = S.Workload("range", 1, 4, 128, 12, 16, 2, 3, 1, 1, 77, (1, 1, 1, 1))


def shaped_inputs(w, cur):
    """Head 0: unit variance, except every 7th query row scaled by 40 (its work
    groups overflow, the others do not).  Head 1: Q scaled by 40 (logits of
    ~60 log2 units spread: overflow).  Head 2: Q[:, 0] = 30, K[:, 0] = -30
    (logits near -115 log2 units: underflow).  Head 3: Q scaled by 6 and the
    keys by a ramp 1 -> 5 over the window (the max grows late; early window
    blocks stay in range, late ones overflow)."""
    q, k, v = S.gen_layer(w, 0, cur)
    qf, kf = S.bf16_bits_to_f32(q).copy(), S.bf16_bits_to_f32(k).copy()
    qf[0, ::7] *= 40.0
    qf[1] *= 40.0
    qf[2, :, 0] = 30.0
    kf[2, :, 0] = -30.0
    qf[3] *= 6.0
    nk = kf.shape[1]
    kf[3] *= (1.0 + 4.0 * np.arange(nk) / max(nk - 1, 1))[:, None].astype(np.float32)
    return S.f32_to_bf16_bits(qf), S.f32_to_bf16_bits(kf), v


@pytest.mark.parametrize("types", [(3, 3, 3, 3), (2, 2, 2, 2), (0, 1, 2, 3), (3, 0, 1, 3)])
@pytest.mark.parametrize("cur", [0, 2, 4])
def test_dynamic_range(hc, types, cur):
    import torch
    w = W_RANGE
    types = np.array(types, np.uint8)
    q, k, v = shaped_inputs(w, cur)
    print(f"dynamic range types={types.tolist()} cur={cur}", flush=True)
    ctx = hc.Context(hc.config_from_workload(w), 0)
    ctx.set_head_types(0, types, cur, dev_bf16(k), dev_bf16(v))
    o = out_tensor(w)
    ctx.attention(0, dev_bf16(q), types, o)
    torch.cuda.synchronize()
    ref = O.routed_attention(types, q, k, v, w.grid_h, w.grid_w, w.frames_per_block,
                             w.spatial_radius)
    assert_close(o.cpu().numpy(), ref, f"dynamic range types={types.tolist()} cur={cur}")
