"""Memory accounting and per-launch timing through the C ABI.

hc_memory_bytes must move by exactly the compact buffers' size when a head table
is replaced: Global heads keep the whole window (round_up(W L, 64) + 64 keys), Sink
and Dummy heads one block (round_up(L, 64) + 64 keys; each head's region ends with one
spare tile that a unit's last 64-key tile may read), K and V in bf16 (Sec. 4.3's
memory saving).  hc_profile_read must count every launch of each kind made while
profiling is on, report a positive duration, and reset on read."""
import numpy as np
import pytest

from helpers import dev_bf16, out_tensor
from synth import inputs as S

pytestmark = pytest.mark.gpu


def round_up(x, m):
    return (x + m - 1) // m * m


def test_memory_bytes_follow_the_head_table(hc):
    w = S.WORKLOADS["tiny"]
    W, L, H, d = w.window_blocks, w.block_tokens, w.n_heads, w.head_dim
    ctx = hc.Context(hc.config_from_workload(w), 0)
    _, k, v = S.gen_layer(w, 0, W - 1)
    base = ctx.memory_bytes()
    ctx.set_head_types(0, np.full(H, S.GLOBAL, np.uint8), W - 1, dev_bf16(k), dev_bf16(v))
    all_global = ctx.memory_bytes()
    g_keys = round_up(W * L, 64) + 64
    sd_keys = round_up(L, 64) + 64
    kv = lambda keys: 2 * keys * d * 2          # K and V of one head, bf16
    assert all_global - base >= H * kv(g_keys)
    mixed = np.array([S.GLOBAL] + [S.SINK] * (H - 1), np.uint8)
    ctx.set_head_types(0, mixed, W - 1, dev_bf16(k), dev_bf16(v))
    assert all_global - ctx.memory_bytes() == (H - 1) * (kv(g_keys) - kv(sd_keys))


def test_profile_counts_every_launch_and_resets(hc):
    import torch
    w = S.WORKLOADS["tiny"]
    W = w.window_blocks
    types = S.head_types(w)[0]                   # one head of each archetype
    ctx = hc.Context(hc.config_from_workload(w), 0)
    q, k, v = S.gen_layer(w, 0, W - 1)
    ctx.set_head_types(0, types, W - 1, dev_bf16(k), dev_bf16(v))
    o = out_tensor(w)
    kb = dev_bf16(k[:, -w.block_tokens:].copy())
    vb = dev_bf16(v[:, -w.block_tokens:].copy())
    ctx.attention(0, dev_bf16(q), types, o)      # builds the work list, not profiled
    torch.cuda.synchronize()
    for kind in (hc.K_DENSE, hc.K_SPATIAL, hc.K_SCATTER, hc.K_COMBINE):
        ctx.profile_read(kind)
    ctx.profile_enable(True)
    steps = 3
    for _ in range(steps):
        ctx.append_block(0, W - 1, kb, vb)
        ctx.attention(0, dev_bf16(q), types, o)
    torch.cuda.synchronize()
    ctx.profile_enable(False)
    for kind in (hc.K_DENSE, hc.K_SPATIAL, hc.K_SCATTER, hc.K_COMBINE):
        ms, n = ctx.profile_read(kind)
        assert n == steps, (kind, n)
        assert ms > 0.0, (kind, ms)
        assert ctx.profile_read(kind) == (0.0, 0)    # read resets
    ctx.attention(0, dev_bf16(q), types, o)      # profiling off: nothing counted
    torch.cuda.synchronize()
    assert ctx.profile_read(hc.K_DENSE) == (0.0, 0)
