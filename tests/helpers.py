"""Shared helpers of the GPU tests: moving seeded bf16 inputs to the device and
comparing GPU outputs with the oracle."""
import numpy as np

MAX_ABS = 1e-2     # tolerance on attention outputs (unit-variance inputs, s = 1/sqrt(d))
MEAN_ABS = 1e-3


def dev_bf16(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def out_tensor(w):
    import torch
    return torch.full((w.n_heads, w.block_tokens, w.head_dim), float("nan"),
                      dtype=torch.float32, device="cuda")


def assert_close(got, ref, what=""):
    got = np.asarray(got, dtype=np.float64)
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    err = np.abs(got - ref)
    print(f"{what}: max|err| {err.max():.3e} mean|err| {err.mean():.3e}", flush=True)
    assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS, (what, err.max(), err.mean())


def stratified_rows(w, n_random=512, seed=0):
    """Query rows covering every frame's four corners, edge midpoints and
    border-adjacent positions, plus seeded random rows (>= 512 in total)."""
    Hg, Wg, F = w.grid_h, w.grid_w, w.frames_per_block
    P = Hg * Wg
    pts = set()
    for f in range(F):
        for y in (0, 1, w.spatial_radius, Hg // 2, Hg - 1 - w.spatial_radius, Hg - 2, Hg - 1):
            for x in (0, 1, 3, 4, 7, 8, w.spatial_radius, Wg // 2, Wg - 1 - w.spatial_radius,
                      Wg - 2, Wg - 1):
                if 0 <= y < Hg and 0 <= x < Wg:
                    pts.add(f * P + y * Wg + x)
    rng = np.random.default_rng(seed)
    pts.update(rng.choice(w.block_tokens, size=n_random, replace=False).tolist())
    return np.array(sorted(pts))
