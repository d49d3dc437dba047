"""Classification + routing at 720P shapes (30 layers x 12 heads, planted
archetypes): hc_classify_heads must reproduce the oracle's labels bit for bit
(stored by tests/golden/make_classify720p.py, which calls only the oracle), then
append + attention run for 4 more blocks and match the oracle on sampled rows."""
import json
import os

import numpy as np
import pytest

from helpers import assert_close, dev_bf16, out_tensor, stratified_rows
from oracle import headcast_oracle as O
from synth import inputs as S

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "classify720p.json")
W = S.WORKLOADS["classify720p"]
CUR = W.window_blocks - 1


@pytest.fixture(scope="module")
def golden():
    if not os.path.exists(GOLDEN):
        pytest.skip("oracle labels not generated: run tests/golden/make_classify720p.py")
    data = json.load(open(GOLDEN))
    if sorted(int(k) for k in data["layers"]) != list(range(W.n_layers)):
        pytest.skip("oracle labels incomplete: run tests/golden/make_classify720p.py")
    return data


@pytest.fixture(scope="module")
def ctx(hc):
    return hc.Context(hc.config_from_workload(W), 0)


@pytest.mark.parametrize("group", range(6))
def test_labels_match_oracle(hc, ctx, golden, group):
    for layer in range(5 * group, 5 * group + 5):
        q, k, v = S.gen_layer(W, layer, CUR, classify_block=CUR)
        labels, stats = ctx.classify_heads(layer, CUR, dev_bf16(q), dev_bf16(k), dev_bf16(v))
        ref = golden["layers"][str(layer)]
        ref_stats = np.array(ref["stats"])
        print(f"layer {layer}: gpu {list(labels)} oracle {ref['labels']}", flush=True)
        assert list(labels) == ref["labels"]
        assert list(labels) == ref["planted"]
        np.testing.assert_allclose(stats[:, :4], ref_stats[:, :4], atol=2e-3)
        np.testing.assert_allclose(stats[:, 4], ref_stats[:, 4], rtol=2e-2, atol=1e-6)
        np.testing.assert_allclose(stats[:, 5], ref_stats[:, 5], atol=3e-3)
        hs, ring = ctx.get_layout(layer)
        assert list(hs) == O.head_slots(labels)
        assert list(ring) == O.ring_slots_of_logical(CUR, W.window_blocks)


def test_routing_after_classification(hc, golden):
    import torch
    layer = 3
    c = hc.Context(hc.config_from_workload(W, n_layers=1), 0)
    q, k, v = S.gen_layer(W, layer, CUR, classify_block=CUR)
    labels, _ = c.classify_heads(0, CUR, dev_bf16(q), dev_bf16(k), dev_bf16(v))
    assert list(labels) == golden["layers"][str(layer)]["labels"]
    rows = stratified_rows(W, n_random=256, seed=5)
    for b in range(CUR + 1, CUR + 5):
        qb, kb, vb = S.gen_step_block(W, layer, b, classify_block=CUR)
        c.append_block(0, b, dev_bf16(kb), dev_bf16(vb))
        o = out_tensor(W)
        c.attention(0, dev_bf16(qb), labels, o)
        torch.cuda.synchronize()
        _, kw, vw = S.gen_layer(W, layer, b, classify_block=CUR)
        ref = O.routed_attention(labels, qb, kw, vw, W.grid_h, W.grid_w, W.frames_per_block,
                                 W.spatial_radius, rows=rows)
        assert_close(o.cpu().numpy()[:, rows], ref, f"classify720p block {b}")
