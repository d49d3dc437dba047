"""GPU parity at logit magnitudes far from unit variance.  The dense and Spatial
kernels first run a pass with the softmax offset fixed at 0 and fall back to the
running-max pass when a row sum leaves [2^-60, 2^96] (overflow or underflow of
2^x); these inputs drive both branches, the merge of per-block Global partials
and of split Spatial partials produced by different passes.  The oracle is the
plain fp64 definition (max subtracted), so any magnitude is exact there.
Tolerance as elsewhere: max-abs 1e-2, mean-abs 1e-3."""
import math

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


# d = 128, 12 x 16 grid, 2 frames per block (L = 384), a full window of 7 blocks
# (7 partials per Global merge), r = 1: the Spatial work of one or two heads is
# split over the 14 key frames (8 partials per Spatial merge)
W_BIGV = S.Workload("bigv", 1, 4, 128, 12, 16, 2, 7, 1, 1, 79, (1, 1, 1, 1))


def big_v_inputs(w, cur, lam_global, lam_spatial, v_scale):
    """Logits equal for every key of a head (Q and K along the first dimension
    only), so every probability of the fixed-offset pass is 2^lam, and V around
    v_scale: a block partial of a Global head then holds about L 2^lam v_scale
    and a split Spatial partial about (keys of 1-2 frames) 2^lam v_scale.  The
    defaults put each partial just below 2^126 -- accepted by a 2^126 bound --
    while the sum of 7 (Global) or 8 (Spatial) of them exceeds fp32's range."""
    q, k, v = S.gen_layer(w, 0, cur)
    d = w.head_dim
    qf = np.zeros(S.bf16_bits_to_f32(q).shape, np.float32)
    kf = np.zeros(S.bf16_bits_to_f32(k).shape, np.float32)
    qf[:, :, 0] = 32.0
    s_log2 = 1.4426950408889634 / math.sqrt(d)
    for h, lam in enumerate([lam_global, lam_spatial, lam_global, lam_spatial]):
        kf[h, :, 0] = S.bf16_bits_to_f32(S.f32_to_bf16_bits(
            np.array([lam / (32.0 * s_log2)], np.float32)))[0]
    vf = v_scale * (1.0 + 0.25 * S.bf16_bits_to_f32(v))
    return S.f32_to_bf16_bits(qf), S.f32_to_bf16_bits(kf), S.f32_to_bf16_bits(vf.astype(np.float32))


@pytest.mark.parametrize("types", [(3, 2, 3, 2), (3, 3, 2, 1)])
def test_large_v_merges_stay_finite(hc, types):
    """Global heads: 7 block partials of about 2^125.3 each; Spatial heads: up to
    8 split partials of about 2^125.5.  Each partial passes a bound of 2^126 on
    its own; their fp32 sum would overflow.  The fixed-offset pass therefore
    accepts only accumulators below 2^121 and reruns the others with the
    running max.  Outputs are compared after dividing by the V scale (2^30)."""
    import torch
    w = W_BIGV
    cur = w.window_blocks - 1
    types = np.array(types, np.uint8)
    v_scale = 2.0 ** 30
    q, k, v = big_v_inputs(w, cur, 86.7, 91.3, v_scale)
    print(f"large-V merges types={types.tolist()}", flush=True)
    ctx = hc.Context(hc.config_from_workload(w), 0)
    ctx.set_head_types(0, types, cur, dev_bf16(k), dev_bf16(v))
    o = out_tensor(w)
    ctx.attention(0, dev_bf16(q), types, o)
    torch.cuda.synchronize()
    ref = O.routed_attention(types, q, k, v, w.grid_h, w.grid_w, w.frames_per_block,
                             w.spatial_radius)
    assert_close(o.cpu().numpy() / v_scale, ref / v_scale, f"large-V merges types={types.tolist()}")


@pytest.mark.parametrize("types", [(3, 0, 1, 2), (3, 3, 3, 3), (0, 1, 0, 1)])
def test_many_overflowed_probabilities_per_row(hc, types):
    """Q scaled by 100 over a full 7-block window: logits of ~144 log2 units
    standard deviation put about a fifth of the keys of every row above 2^128,
    dozens per 384-key unit.  The fixed-offset pass then holds infinite
    probabilities, accumulators in which +inf meets -inf (NaN in practically
    every element, so no element is a finite or infinite witness) and row sums
    that meet the zeros of the row-sum selector (NaN).  Every such group must
    fail the acceptance test and rerun with the running max; the outputs are
    compared in full with the oracle."""
    import torch
    w = W_BIGV
    cur = w.window_blocks - 1
    types = np.array(types, np.uint8)
    q, k, v = S.gen_layer(w, 0, cur)
    q = S.f32_to_bf16_bits(S.bf16_bits_to_f32(q) * np.float32(100.0))
    print(f"overflowed rows types={types.tolist()}", flush=True)
    ctx = hc.Context(hc.config_from_workload(w), 0)
    ctx.set_head_types(0, types, cur, dev_bf16(k), dev_bf16(v))
    o = out_tensor(w)
    ctx.attention(0, dev_bf16(q), types, o)
    torch.cuda.synchronize()
    ref = O.routed_attention(types, q, k, v, w.grid_h, w.grid_w, w.frames_per_block,
                             w.spatial_radius)
    assert_close(o.cpu().numpy(), ref, f"overflowed rows types={types.tolist()}")
