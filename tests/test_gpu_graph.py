"""The routed denoising step (append of the current block + attention, every layer)
captured once into a HIP graph and replayed.  After one call at the same window fill the
library only enqueues kernels on the caller's stream, so such a step can be captured.
Each replay runs on new inputs copied into the captured buffers, with the program's own
eager library calls and synchronisations between replays, and must equal an eager step
on the same inputs bit for bit (same kernels and work lists, no atomics); one replay is
also checked against the oracle."""
import numpy as np
import pytest

from helpers import assert_close, dev_bf16
from oracle import headcast_oracle as O
from synth import inputs as S

pytestmark = pytest.mark.gpu


def test_graph_replay_of_routed_steps(hc):
    import torch
    # 2 layers x 8 heads, grid 12 x 16, 3 frames per block, window of 4 blocks, r = 2
    w = S.Workload("graph", 2, 8, 128, 12, 16, 3, 4, 2, 2, 4242, (4, 4, 4, 4))
    W, L, NL, H, d = w.window_blocks, w.block_tokens, w.n_layers, w.n_heads, w.head_dim
    tables = [np.array(t, np.uint8) for t in ([0, 1, 2, 3, 3, 2, 1, 0], [3, 3, 2, 2, 1, 0, 3, 2])]
    cur = W + 1                                   # window full, ring already wrapped once
    ctx = hc.Context(hc.config_from_workload(w), 0)
    win = [S.gen_layer(w, l, cur) for l in range(NL)]
    for l in range(NL):
        ctx.set_head_types(l, tables[l], cur, dev_bf16(win[l][1]), dev_bf16(win[l][2]))

    # captured buffers: the step's query and current block of every layer, and its outputs
    q_buf = [torch.empty((H, L, d), dtype=torch.bfloat16, device="cuda") for _ in range(NL)]
    k_buf = [torch.empty_like(q_buf[0]) for _ in range(NL)]
    v_buf = [torch.empty_like(q_buf[0]) for _ in range(NL)]
    o_buf = [torch.empty((H, L, d), dtype=torch.float32, device="cuda") for _ in range(NL)]
    rng = np.random.default_rng(77)

    def load_inputs():
        """New q and current-block K/V (bf16 bits of N(0,1)) into the captured buffers."""
        host = []
        for l in range(NL):
            q, k, v = (S.f32_to_bf16_bits(rng.standard_normal((H, L, d)).astype(np.float32))
                       for _ in range(3))
            q_buf[l].copy_(dev_bf16(q)); k_buf[l].copy_(dev_bf16(k)); v_buf[l].copy_(dev_bf16(v))
            host.append((q, k, v))
        torch.cuda.synchronize()
        return host

    def step():
        for l in range(NL):
            ctx.append_block(l, cur, k_buf[l], v_buf[l])
            ctx.attention(l, q_buf[l], tables[l], o_buf[l])

    load_inputs()
    step()                                        # eager: builds the work lists
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(3):
        host = load_inputs()
        for o in o_buf:
            o.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        got = [o.clone() for o in o_buf]
        for o in o_buf:
            o.fill_(float("nan"))
        step()                                    # eager step on the same inputs
        torch.cuda.synchronize()
        for l in range(NL):
            assert torch.equal(got[l], o_buf[l]), f"replay {rep} layer {l} differs from eager"
        if rep == 1:
            for l in range(NL):
                q, k, v = host[l]
                kw = win[l][1].copy(); vw = win[l][2].copy()
                kw[:, -L:] = k; vw[:, -L:] = v   # the current block, rewritten
                ref = O.routed_attention(tables[l], q, kw, vw, w.grid_h, w.grid_w,
                                         w.frames_per_block, w.spatial_radius)
                assert_close(got[l].cpu().numpy(), ref, f"replay {rep} layer {l}")
