"""Element-wise parity of the classification attention (Sec. 4.2: Eq. 2 and the
three proxies).  The fused sweep gives O_ref as the merge of one partial per
window block and O_sink / O_dummy as the single-block partials of block 0 and of
the current block normalised on their own; the Spatial proxy runs at radius r_p.
All four are read back through hc_classify_outputs and compared with the
oracle's outputs on the same seeded window, element by element, at the
attention tolerance of the other parity tests."""
import math

import numpy as np
import pytest

from helpers import assert_close, dev_bf16, stratified_rows
from oracle import headcast_oracle as O
from synth import inputs as S

pytestmark = pytest.mark.gpu

OUTPUTS = ((O.GLOBAL, "CLS_O_REF"), (O.SINK, "CLS_O_SINK"), (O.DUMMY, "CLS_O_DUMMY"),
           (O.SPATIAL, "CLS_O_SPATIAL"))


def _empty(w):
    import torch
    return torch.full((w.n_heads, w.block_tokens, w.head_dim), float("nan"),
                      dtype=torch.float32, device="cuda")


def _check_outputs(hc, w, heads, rows=None):
    import torch
    cur = w.window_blocks - 1
    q, k, v = S.gen_layer(w, 0, cur)
    ctx = hc.Context(hc.config_from_workload(w), 0)
    o = _empty(w)
    with pytest.raises(hc.HeadCastError) as e:
        ctx.classify_outputs(hc.CLS_O_REF, o)        # nothing classified yet
    assert e.value.status == hc.HC_E_STATE
    ctx.classify_heads(0, cur, dev_bf16(q), dev_bf16(k), dev_bf16(v))
    g = O.Geometry(w.grid_h, w.grid_w, w.frames_per_block, w.window_blocks)
    scale = 1.0 / math.sqrt(w.head_dim)
    for kind, name in OUTPUTS:
        o = _empty(w)
        ctx.classify_outputs(getattr(hc, name), o)
        torch.cuda.synchronize()
        got = o.cpu().numpy()
        assert np.isfinite(got).all(), f"{name}: rows left unwritten"
        for h in heads:
            ref = O.attend_kind(kind, O.widen(q[h]), O.widen(k[h]), O.widen(v[h]), g,
                                w.proxy_radius, scale, rows)
            assert_close(got[h] if rows is None else got[h][rows], ref,
                         f"{w.name} {name} head {h}")
    with pytest.raises(hc.HeadCastError) as e:
        ctx.classify_outputs(4, o)
    assert e.value.status == hc.HC_E_INVAL


def test_classify_outputs_tiny(hc):
    w = S.WORKLOADS["tiny"]
    _check_outputs(hc, w, heads=range(w.n_heads))


def test_classify_outputs_tiny_planted(hc):
    w = S.WORKLOADS["tiny_planted"]
    _check_outputs(hc, w, heads=range(w.n_heads))


def test_classify_outputs_480p_sampled_rows(hc):
    """480P (L = 4680: a ragged last query tile, seven block partials per row),
    every output on stratified rows of three heads."""
    w = S.WORKLOADS["480p"]
    _check_outputs(hc, w, heads=(0, 5, 11), rows=stratified_rows(w))
