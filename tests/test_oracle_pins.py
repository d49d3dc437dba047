"""Pins for the CPU oracle: every check compares the oracle against something
other than itself -- a library routine (torch SDPA in float64), a closed form,
an invariant of the method, brute force on tiny inputs, or a number the paper
prints."""
import math

import numpy as np
import pytest
import torch

from oracle import headcast_oracle as O
from synth import inputs as S

SDPA = torch.nn.functional.scaled_dot_product_attention


def sdpa(q, k, v, scale, mask=None):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))[None, None]
    m = None if mask is None else torch.from_numpy(mask)
    return SDPA(t(q), t(k), t(v), attn_mask=m, scale=scale)[0, 0].numpy()


def tiny_layer(cur_block=3, seed_w="tiny"):
    w = S.WORKLOADS[seed_w]
    q, k, v = S.gen_layer(w, 0, cur_block)
    return w, O.widen(q), O.widen(k), O.widen(v)


def geom(w, n):
    return O.Geometry(w.grid_h, w.grid_w, w.frames_per_block, n)


# --- P1 / P2: Global, Sink and Dummy against the library routine -----------------
@pytest.mark.parametrize("kind", [O.GLOBAL, O.SINK, O.DUMMY])
def test_dense_kinds_match_sdpa(kind):
    w, q, k, v = tiny_layer()
    g = geom(w, 4)
    s = 1 / math.sqrt(w.head_dim)
    L = w.block_tokens
    sl = {O.GLOBAL: slice(0, 4 * L), O.SINK: slice(0, L), O.DUMMY: slice(3 * L, 4 * L)}[kind]
    for h in range(w.n_heads):
        got = O.attend_kind(kind, q[h], k[h], v[h], g, 1, s)
        ref = sdpa(q[h], k[h][sl], v[h][sl], s)
        np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_global_480p_slice_matches_sdpa():
    w = S.WORKLOADS["480p"]
    L = w.block_tokens
    q = O.widen(S.gen_block(w, 0, 0, S.T_Q, 6))[:256]
    k = np.concatenate([O.widen(S.gen_block(w, 0, 0, S.T_K, b)) for b in range(7)])
    v = np.concatenate([O.widen(S.gen_block(w, 0, 0, S.T_V, b)) for b in range(7)])
    s = 1 / math.sqrt(128)
    got = O.attend_shared(q, k, v, s)
    np.testing.assert_allclose(got, sdpa(q, k, v, s), rtol=0, atol=1e-12)
    assert k.shape[0] == 7 * L


def test_attend_one_matches_sdpa_and_shared():
    w, q, k, v = tiny_layer()
    s = 0.37
    idx = np.array([5, 9, 100, 511, 3])
    got = O.attend_one(q[0][7], k[0], v[0], idx, s)
    ref = sdpa(q[0][7:8], k[0][idx], v[0][idx], s)[0]
    np.testing.assert_allclose(got, ref, atol=1e-13)


# --- P3: a Spatial window covering the frame equals Global -------------------------
@pytest.mark.parametrize("cur_block", [1, 3])
def test_spatial_full_frame_equals_global(cur_block):
    w, q, k, v = tiny_layer(cur_block)
    n = k.shape[1] // w.block_tokens
    g = geom(w, n)
    s = 1 / math.sqrt(w.head_dim)
    r = max(w.grid_h, w.grid_w) - 1
    for h in range(w.n_heads):
        a = O.attend_kind(O.SPATIAL, q[h], k[h], v[h], g, r, s)
        b = O.attend_kind(O.GLOBAL, q[h], k[h], v[h], g, r, s)
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


# --- P4: r = 0 sees exactly the same position in every window frame --------------
def test_spatial_r0_closed_form_slice():
    w, q, k, v = tiny_layer()
    g = geom(w, 4)
    s = 1 / math.sqrt(w.head_dim)
    out = O.attend_kind(O.SPATIAL, q[2], k[2], v[2], g, 0, s)
    P = w.tokens_per_frame
    for t in [0, 7, 8, 63, 64, 100, 127]:
        idx = (t % P) + P * np.arange(4 * w.frames_per_block)
        ref = sdpa(q[2][t:t + 1], k[2][idx], v[2][idx], s)[0]
        np.testing.assert_allclose(out[t], ref, atol=1e-12)


# --- P5: Spatial against a materialised boolean mask + SDPA ------------------------
@pytest.mark.parametrize("r", [1, 2, 3])
def test_spatial_matches_materialised_mask(r):
    w, q, k, v = tiny_layer()
    L, P, Wg = w.block_tokens, w.tokens_per_frame, w.grid_w
    n = 4
    mask = np.zeros((L, n * L), dtype=bool)
    for t in range(L):                       # brute force over coordinates
        y, x = divmod(t % P, Wg)
        for j in range(n * L):
            y2, x2 = divmod(j % P, Wg)
            mask[t, j] = abs(y2 - y) <= r and abs(x2 - x) <= r
    s = 1 / math.sqrt(w.head_dim)
    got = O.attend_kind(O.SPATIAL, q[2], k[2], v[2], geom(w, n), r, s)
    np.testing.assert_allclose(got, sdpa(q[2], k[2], v[2], s, mask), atol=1e-12)


def test_spatial_ragged_grid_matches_mask():
    # a grid whose width is not a multiple of anything convenient
    Hg, Wg, F, n, d, r = 5, 7, 3, 2, 16, 2
    L, P = F * Hg * Wg, Hg * Wg
    rng = np.random.default_rng(5)
    q, k, v = rng.standard_normal((L, d)), rng.standard_normal((n * L, d)), rng.standard_normal((n * L, d))
    mask = np.zeros((L, n * L), dtype=bool)
    for t in range(L):
        y, x = divmod(t % P, Wg)
        for j in range(n * L):
            y2, x2 = divmod(j % P, Wg)
            mask[t, j] = abs(y2 - y) <= r and abs(x2 - x) <= r
    got = O.attend_kind(O.SPATIAL, q, k, v, O.Geometry(Hg, Wg, F, n), r, 0.25)
    np.testing.assert_allclose(got, sdpa(q, k, v, 0.25, mask), atol=1e-12)
    rows = np.array([0, 6, 34, 35, 104])
    part = O.attend_spatial(q, k, v, O.Geometry(Hg, Wg, F, n), r, 0.25, rows)
    np.testing.assert_allclose(part, got[rows], atol=1e-13)


# --- P6: fingerprint -- Q = 0 gives the plain mean of V over the key set ----------
def test_fingerprint_uniform_weights():
    w = S.WORKLOADS["tiny"]
    Hg, Wg, F, n, r = w.grid_h, w.grid_w, w.frames_per_block, 3, 1
    L, P = w.block_tokens, w.tokens_per_frame
    j = np.arange(n * L)
    V = np.stack([np.ones(n * L), (j % P) // Wg, (j % P) % Wg, j // P, j // L], axis=1).astype(float)
    K = np.random.default_rng(1).standard_normal((n * L, 5))
    Q = np.zeros((L, 5))
    g = O.Geometry(Hg, Wg, F, n)

    def clip_mean(i, N):
        lo, hi = max(0, i - r), min(N - 1, i + r)
        return (lo + hi) / 2

    out = O.attend_kind(O.SPATIAL, Q, K, V, g, r, 1.0)
    for t in range(L):
        y, x = divmod(t % P, Wg)
        np.testing.assert_allclose(out[t], [1, clip_mean(y, Hg), clip_mean(x, Wg),
                                            (n * F - 1) / 2, (n - 1) / 2], atol=1e-12)
    sink = O.attend_kind(O.SINK, Q, K, V, g, r, 1.0)
    dummy = O.attend_kind(O.DUMMY, Q, K, V, g, r, 1.0)
    glob = O.attend_kind(O.GLOBAL, Q, K, V, g, r, 1.0)
    np.testing.assert_allclose(sink[:, 3:], np.tile([(F - 1) / 2, 0], (L, 1)), atol=1e-12)
    np.testing.assert_allclose(dummy[:, 3:], np.tile([(n - 1) * F + (F - 1) / 2, n - 1], (L, 1)), atol=1e-12)
    np.testing.assert_allclose(glob[:, 3:], np.tile([(n * F - 1) / 2, (n - 1) / 2], (L, 1)), atol=1e-12)


# --- P7: linearity in V -----------------------------------------------------------
@pytest.mark.parametrize("kind", [O.SINK, O.DUMMY, O.SPATIAL, O.GLOBAL])
def test_linearity_in_v(kind):
    w, q, k, v = tiny_layer()
    g = geom(w, 4)
    s = 1 / math.sqrt(w.head_dim)
    a, c = -2.5, 0.75
    o1 = O.attend_kind(kind, q[1], k[1], v[1], g, 1, s)
    o2 = O.attend_kind(kind, q[1], k[1], a * v[1] + c, g, 1, s)
    np.testing.assert_allclose(o2, a * o1 + c, atol=1e-12)


# --- P8: key order does not matter (logical vs physical ring order) ---------------
def test_permutation_invariance_ring_order():
    w, q, k, v = tiny_layer(cur_block=5)
    L = w.block_tokens
    slots = O.ring_slots_of_logical(5, 4)               # logical -> physical
    phys_k = np.empty_like(k[3]); phys_v = np.empty_like(v[3])
    for i, sl in enumerate(slots):
        phys_k[sl * L:(sl + 1) * L] = k[3][i * L:(i + 1) * L]
        phys_v[sl * L:(sl + 1) * L] = v[3][i * L:(i + 1) * L]
    s = 1 / math.sqrt(w.head_dim)
    a = O.attend_shared(q[3], k[3], v[3], s)
    b = O.attend_shared(q[3], phys_k, phys_v, s)
    np.testing.assert_allclose(a, b, atol=1e-12)


# --- P9: classification special cases ---------------------------------------------
def _classify(q, k, v, w, rp=2):
    return O.classify_layer(q, k, v, w.grid_h, w.grid_w, w.frames_per_block, rp)


def test_constant_v_gives_sink():
    w = S.WORKLOADS["tiny"]
    q, k, v = S.gen_layer(w, 0, 3)
    v = np.full_like(v, S.f32_to_bf16_bits(np.array([1.5], np.float32))[0])
    labels, st = _classify(q, k, v, w)
    assert (labels == O.SINK).all()
    np.testing.assert_allclose(st[:, :4], 1.0, atol=1e-12)
    np.testing.assert_allclose(st[:, 4], 0.0, atol=1e-24)


def _shifted(w, boost_block):
    q, k, v = S.gen_layer(w, 0, 3)
    kf = S.bf16_bits_to_f32(k)
    L = w.block_tokens
    # keys outside the boosted block are pushed away from every query:
    # a strong negative shift along q's mean direction makes their weight ~0
    qm = S.bf16_bits_to_f32(q).mean(1, keepdims=True)            # [H][1][d]
    qn = qm / np.linalg.norm(qm, axis=2, keepdims=True)
    sel = np.ones(kf.shape[1], dtype=bool)
    sel[boost_block * L:(boost_block + 1) * L] = False
    qf = S.bf16_bits_to_f32(q) + 8 * qn                          # queries share a direction
    kf[:, sel] -= 40 * qn[:, 0][:, None, :]
    return S.f32_to_bf16_bits(qf), S.f32_to_bf16_bits(kf), v


def test_negative_shift_outside_block0_gives_sink():
    w = S.WORKLOADS["tiny"]
    labels, st = _classify(*_shifted(w, 0), w)
    assert (labels == O.SINK).all(), st


def test_negative_shift_outside_current_gives_dummy():
    w = S.WORKLOADS["tiny"]
    labels, st = _classify(*_shifted(w, 3), w)
    assert (labels == O.DUMMY).all(), st


def test_full_frame_proxy_gives_spatial_for_unbiased_heads():
    w = S.WORKLOADS["tiny"]
    q, k, v = S.gen_layer(w, 0, 3)
    labels, st = _classify(q, k, v, w, rp=7)
    np.testing.assert_allclose(st[:, 2], 1.0, atol=1e-12)
    np.testing.assert_allclose(st[:, 5], 1.0, atol=1e-12)
    for h in range(4):
        if st[h, 0] < O.THETA and st[h, 1] < O.THETA:
            assert labels[h] == O.SPATIAL


def test_decide_hierarchy_and_inclusive_thresholds():
    T, C = O.THETA, O.THETA_SCORE
    assert O.decide([T, 1, 1, 1, 0, 1]) == O.SINK           # Sink has priority
    assert O.decide([T - 1e-9, T, 1, 1, 0, 1]) == O.DUMMY
    assert O.decide([0, T - 1e-9, T, 0, 0, C]) == O.SPATIAL  # score exactly at threshold
    assert O.decide([0, 0, T, 0, 0, C - 1e-9]) == O.GLOBAL
    assert O.decide([0, 0, T - 1e-9, 0, 0, 1]) == O.GLOBAL


# --- P10: percentile convention ----------------------------------------------------
def test_percentile5_matches_numpy_and_hand_values():
    rng = np.random.default_rng(3)
    for n in [1, 2, 3, 20, 21, 101, 10800]:
        x = rng.random(n)
        assert O.percentile5(x) == pytest.approx(np.percentile(x, 5), abs=1e-15)
    # 21 values 0..20: rank 0.05 * 20 = 1 -> exactly the second smallest
    assert O.percentile5(np.arange(21)[::-1]) == 1.0
    # 11 values 0..10: rank 0.5 -> halfway between 0 and 1
    assert O.percentile5(np.arange(11)) == 0.5


def test_p5_flip_when_nonlocal_tokens_cross_rank():
    # 101 token cosines: k bad tokens at 0.0, the rest at 1.0.  rank = 5.0
    base = np.ones(101)
    for kbad, want in [(5, 1.0), (6, 0.0)]:
        x = base.copy(); x[:kbad] = 0.0
        assert O.percentile5(x) == want


# --- P11: the MSE term of the spatial score ------------------------------------------
def test_mse_scales_quadratically_and_cos_invariant():
    rng = np.random.default_rng(11)
    ref, sp = rng.standard_normal((50, 8)), rng.standard_normal((50, 8))
    s1 = O.head_statistics(ref, ref, ref, sp)
    c = 3.0
    s2 = O.head_statistics(c * ref, c * ref, c * ref, c * sp)
    np.testing.assert_allclose(s2[:4], s1[:4], atol=1e-14)
    assert s2[4] == pytest.approx(c * c * s1[4], rel=1e-14)
    # exact mean of squared differences
    assert s1[4] == pytest.approx(((sp - ref) ** 2).sum() / 400, rel=1e-14)


def test_spatial_to_global_flip_point():
    # a head whose spatial proxy is almost right: cos stays >= theta, the MSE grows
    # as c^2 when V is scaled by c; the label flips at c* = sqrt((P5 - theta_sc)/(gamma MSE_1))
    rng = np.random.default_rng(2)
    ref = rng.standard_normal((200, 16))
    sp = ref + 0.05 * rng.standard_normal((200, 16))
    far = rng.standard_normal((200, 16))
    st = O.head_statistics(ref, far, far, sp)
    assert st[2] >= O.THETA and st[0] < O.THETA and st[1] < O.THETA
    cstar = math.sqrt((st[3] - O.THETA_SCORE) / (O.GAMMA * st[4]))
    lo = O.head_statistics(ref * cstar * 0.999, far, far, sp * cstar * 0.999)
    hi = O.head_statistics(ref * cstar * 1.001, far, far, sp * cstar * 1.001)
    assert O.decide(lo) == O.SPATIAL and O.decide(hi) == O.GLOBAL


def test_token_cos_zero_vector():
    a = np.zeros((2, 4)); b = np.ones((2, 4))
    assert (O.token_cos(a, b) == 0).all()
    np.testing.assert_allclose(O.token_cos(b, 2 * b), 1.0)


# --- Eq. 3 / Eq. 4: cosines are taken per token, then averaged (or ranked) --------------
def test_cos_mean_is_over_token_cosines_hand_values():
    # Three tokens, d = 2, O_ref = (1, 0) for each.  Proxy tokens at angle 0, 90 and
    # 180 degrees (lengths 2, 3, 1): token cosines 1, 0, -1, so the Eq. 3 mean is 0.
    # One cosine of the flattened [3][2] outputs would be (2 + 0 - 1) / (sqrt 3 sqrt 14)
    # = 1 / sqrt 42, and cosines along the other axis (per dimension over the tokens)
    # average to 1 / (2 sqrt 15): neither is 0.
    ref = np.array([[1.0, 0.0], [1.0, 0.0], [1.0, 0.0]])
    sp = np.array([[2.0, 0.0], [0.0, 3.0], [-1.0, 0.0]])
    # the other proxies: token cosines (1, 1, 0) -> mean 2/3 and (0, -1, -1) -> mean -2/3
    sink = np.array([[5.0, 0.0], [0.5, 0.0], [0.0, -7.0]])
    dummy = np.array([[0.0, 4.0], [-2.0, 0.0], [-3.0, 0.0]])
    st = O.head_statistics(ref, sink, dummy, sp)
    assert st[0] == pytest.approx(2.0 / 3.0, abs=1e-15)
    assert st[1] == pytest.approx(-2.0 / 3.0, abs=1e-15)
    assert st[2] == 0.0
    # P5 over the three token cosines (-1, 0, 1): rank 0.05 * 2 = 0.1 -> -1 + 0.1 * 1
    assert st[3] == pytest.approx(-0.9, abs=1e-15)
    # MSE over all 6 elements: (1 + 0 + 1 + 9 + 4 + 0) / 6
    assert st[4] == pytest.approx(15.0 / 6.0, abs=1e-15)
    assert st[5] == pytest.approx(-0.9 - O.GAMMA * 2.5, abs=1e-14)


def test_p5_is_over_token_cosines_hand_values():
    # 21 tokens, d = 3, O_ref = (1, 0, 0).  Each proxy token is a Pythagorean
    # direction, so its cosine is an exact ratio: 19 tokens at cos 1 (length 2),
    # one at -3/5 (the smallest) and one at 5/13 (the second smallest).  With 21
    # tokens the 5th-percentile rank is 0.05 * 20 = 1: P5 is exactly 5/13.
    ref = np.tile([1.0, 0.0, 0.0], (21, 1))
    sp = np.tile([2.0, 0.0, 0.0], (21, 1))
    sp[7] = [-3.0, 0.0, 4.0]      # cos -3/5
    sp[13] = [5.0, 12.0, 0.0]     # cos 5/13
    st = O.head_statistics(ref, ref, ref, sp)
    assert st[3] == pytest.approx(5.0 / 13.0, abs=1e-15)
    assert st[2] == pytest.approx((19.0 - 3.0 / 5.0 + 5.0 / 13.0) / 21.0, abs=1e-15)
    # exact MSE: 19 tokens contribute 1 each, the two others (16 + 16) and (16 + 144)
    assert st[4] == pytest.approx((19.0 + 32.0 + 160.0) / 63.0, abs=1e-14)
    # a token moved from the second-smallest cosine to cos 1 moves P5 to the
    # interpolation between -3/5 and 1 at rank 1: exactly 1
    sp[13] = [2.0, 0.0, 0.0]
    assert O.head_statistics(ref, ref, ref, sp)[3] == pytest.approx(1.0, abs=1e-15)


# --- P12: planted archetypes are recovered by brute force -----------------------------
def test_tiny_planted_labels_recovered():
    w = S.WORKLOADS["tiny_planted"]
    q, k, v = S.gen_layer(w, 0, w.window_blocks - 1)
    labels, st = _classify(q, k, v, w, rp=w.proxy_radius)
    assert list(labels) == list(S.head_types(w)[0]), st
    # margins from every threshold the decision looked at
    thr = [O.THETA, O.THETA, O.THETA, None, None, O.THETA_SCORE]
    for h in range(4):
        for i, t in enumerate(thr):
            if t is not None:
                assert abs(st[h, i] - t) > 1e-3


def test_planted_spatial_channels_encode_distance():
    # the coordinate channels reproduce -0.5 * dist^2 (up to a per-query constant)
    w = S.WORKLOADS["tiny_planted"]
    qc = S._spatial_q_channels(w)
    kb = S.f32_to_bf16_bits(S._spatial_k_channels(w).astype(np.float32))
    kc = O.widen(kb)
    qc_b = O.widen(S.f32_to_bf16_bits(qc.astype(np.float32)))
    logit = (qc_b @ kc.T) / math.sqrt(w.head_dim)
    P, Wg = w.tokens_per_frame, w.grid_w
    for t in [0, 9, 27, 63]:
        y, x = divmod(t % P, Wg)
        yy, xx = np.divmod(np.arange(w.block_tokens) % P, Wg)
        want = -0.5 * ((yy - y) ** 2 + (xx - x) ** 2)
        d = logit[t] - want
        assert np.ptp(d) < 5e-3


# --- P13: the paper's cost models -------------------------------------------------------
def test_paper_flop_ratio_table6_480p():
    # Table 6 (480P head counts) -> the ~64% attention-FLOP reduction of Appendix B
    r = O.paper_flop_ratio(1.6, 93.8, 168.2, 96.5, n_total=30 * 12)
    assert r == pytest.approx(0.3635, abs=5e-5)
    assert 1 - r == pytest.approx(0.64, abs=0.005)


def test_paper_kv_reduction():
    # Appendix C: (N_s + N_d) / N ~ 166/360 -> ~34% predicted
    assert O.paper_kv_reduction(166 / 360) == pytest.approx(0.346, abs=5e-4)


def test_paper_cell_fraction_480p():
    # Appendix B: a 10x10 cell is about 1/16 of a 30x52 latent frame
    assert 100 / (30 * 52) == pytest.approx(1 / 16, rel=0.03)


def test_in_set_pairs_brute_force():
    for (Hg, Wg, F, n, r) in [(8, 8, 2, 4, 1), (5, 7, 3, 2, 2), (6, 9, 1, 3, 4)]:
        g = O.Geometry(Hg, Wg, F, n)
        for kind in (O.SINK, O.DUMMY, O.SPATIAL, O.GLOBAL):
            brute = sum(O.key_set(kind, g, t, r).size for t in range(g.L))
            assert O.in_set_pairs(kind, Hg, Wg, F, n, r) == brute


def test_flops_720p_closed_forms():
    L, Lk, d = 10800, 75600, 128
    assert O.algorithmic_flops([O.GLOBAL], 45, 80, 3, 7, 4, d) == 4 * d * L * Lk
    assert O.algorithmic_flops([O.SINK], 45, 80, 3, 7, 4, d) == 4 * d * L * L
    # clipped 9x9 window: rows 9*45-20 = 385, cols 9*80-20 = 700 (per axis sums)
    assert O.in_set_pairs(O.SPATIAL, 45, 80, 3, 7, 4) == 3 * 385 * 700 * 21


# --- P14: layout integers -------------------------------------------------------------------
def test_ring_slots_hand_worked():
    # W = 4: block b >= 1 goes to slot 1 + (b-1) mod 3; logical order = sink, then oldest..current
    assert O.ring_slots_of_logical(0, 4) == [0, -1, -1, -1]
    assert O.ring_slots_of_logical(2, 4) == [0, 1, 2, -1]
    assert O.ring_slots_of_logical(3, 4) == [0, 1, 2, 3]
    assert O.ring_slots_of_logical(4, 4) == [0, 2, 3, 1]
    assert O.ring_slots_of_logical(5, 4) == [0, 3, 1, 2]
    assert O.ring_slots_of_logical(6, 4) == [0, 1, 2, 3]
    for W in (2, 3, 4, 7):
        for b in range(1, 4 * W):
            assert O.simulate_ring(b + 1, W)[b] == 1 + (b - 1) % (W - 1) if W > 1 else 0


def test_window_blocks_matches_input_contract():
    for W in (4, 7):
        for c in range(3 * W):
            assert O.window_blocks(c, W) == S.window_block_ids(c, W)


def test_head_slots():
    assert O.head_slots([0, 1, 2, 3]) == [0, 1, 0, 0]
    assert O.head_slots([3, 1, 3, 0, 2, 2, 1]) == [0, 0, 1, 1, 0, 1, 2]


# --- cell variant of the Spatial path (Sec. 4.4, Sec. 5.1; reading R20) -----------
@pytest.mark.parametrize("N,c,bounds", [
    (45, 10, [0, 10, 20, 30, 40, 45]),      # 4.5 cells -> 5, the last one short
    (52, 10, [0, 10, 20, 30, 40, 52]),      # 5.2 -> 5, the last one absorbs 2
    (30, 10, [0, 10, 20, 30]),
    (68, 10, [0, 10, 20, 30, 40, 50, 60, 68]),
    (120, 10, list(range(0, 121, 10))),
    (8, 3, [0, 3, 6, 8]), (7, 3, [0, 3, 7]), (5, 2, [0, 2, 4, 5]),
    (4, 10, [0, 4]), (8, 20, [0, 8])])      # a cell wider than the frame: one cell
def test_cell_bounds_hand_values(N, c, bounds):
    assert O.cell_bounds(N, c).tolist() == bounds


@pytest.mark.parametrize("c", [2, 3, 5])
def test_cells_match_materialised_mask(c):
    # brute force: the cell of a position is fixed by the hand-listed boundaries
    w, q, k, v = tiny_layer()
    L, P, Wg = w.block_tokens, w.tokens_per_frame, w.grid_w
    edges = {2: [0, 2, 4, 6, 8], 3: [0, 3, 6, 8], 5: [0, 5, 8]}[c]   # 8 / c rounded
    cell_id = lambda i: sum(i >= e for e in edges[1:-1])
    n = 4
    mask = np.zeros((L, n * L), dtype=bool)
    for t in range(L):
        y, x = divmod(t % P, Wg)
        for j in range(n * L):
            y2, x2 = divmod(j % P, Wg)
            mask[t, j] = cell_id(y2) == cell_id(y) and cell_id(x2) == cell_id(x)
    s = 1 / math.sqrt(w.head_dim)
    got = O.attend_kind(O.SPATIAL, q[2], k[2], v[2], geom(w, n), 0, s, cell=c)
    np.testing.assert_allclose(got, sdpa(q[2], k[2], v[2], s, mask), atol=1e-12)
    rows = np.array([0, 9, 27, 63, 64, 127])
    part = O.attend_cells(q[2], k[2], v[2], geom(w, n), c, s, rows)
    np.testing.assert_allclose(part, got[rows], atol=1e-13)


def test_cell_covering_the_frame_equals_global():
    w, q, k, v = tiny_layer(3)
    g = geom(w, 4)
    s = 1 / math.sqrt(w.head_dim)
    for h in range(w.n_heads):
        a = O.attend_kind(O.SPATIAL, q[h], k[h], v[h], g, 0, s, cell=max(w.grid_h, w.grid_w))
        b = O.attend_kind(O.GLOBAL, q[h], k[h], v[h], g, 0, s)
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_cell_fingerprint_uniform_weights():
    # Q = 0: every key of the cell gets the same weight, so O is the mean of V
    # over the cell rows / columns and over all window frames
    Hg, Wg, F, n, c = 7, 9, 2, 3, 3
    L, P = F * Hg * Wg, Hg * Wg
    j = np.arange(n * L)
    V = np.stack([np.ones(n * L), (j % P) // Wg, (j % P) % Wg, j // P], axis=1).astype(float)
    K = np.random.default_rng(2).standard_normal((n * L, 4))
    out = O.attend_kind(O.SPATIAL, np.zeros((L, 4)), K, V, O.Geometry(Hg, Wg, F, n), 0, 1.0,
                        cell=c)
    ey, ex = [0, 3, 7], [0, 3, 6, 9]          # 7/3 -> 2 cells, 9/3 -> 3 cells
    span = lambda i, e: next((e[m], e[m + 1]) for m in range(len(e) - 1) if e[m] <= i < e[m + 1])
    for t in range(L):
        y, x = divmod(t % P, Wg)
        (y0, y1), (x0, x1) = span(y, ey), span(x, ex)
        np.testing.assert_allclose(out[t], [1, (y0 + y1 - 1) / 2, (x0 + x1 - 1) / 2,
                                            (n * F - 1) / 2], atol=1e-12)


# --- two-block Sink / Dummy variant (App. B, App. C; reading R1 alternative) -----
@pytest.mark.parametrize("cur_block", [0, 1, 2, 3, 5])
def test_two_block_sink_dummy_match_sdpa_on_concatenation(cur_block):
    w, q, k, v = tiny_layer(cur_block)
    L = w.block_tokens
    n = k.shape[1] // L
    g = geom(w, n)
    s = 1 / math.sqrt(w.head_dim)
    blk = lambda a, i: a[i * L:(i + 1) * L]
    sink_k = np.concatenate([blk(k[0], 0)] + ([blk(k[0], n - 1)] if n >= 2 else []))
    sink_v = np.concatenate([blk(v[0], 0)] + ([blk(v[0], n - 1)] if n >= 2 else []))
    dum_k = np.concatenate(([blk(k[1], n - 2)] if n >= 2 else []) + [blk(k[1], n - 1)])
    dum_v = np.concatenate(([blk(v[1], n - 2)] if n >= 2 else []) + [blk(v[1], n - 1)])
    got_s = O.attend_kind(O.SINK, q[0], k[0], v[0], g, 1, s, sd_blocks=2)
    got_d = O.attend_kind(O.DUMMY, q[1], k[1], v[1], g, 1, s, sd_blocks=2)
    np.testing.assert_allclose(got_s, sdpa(q[0], sink_k, sink_v, s), atol=1e-12)
    np.testing.assert_allclose(got_d, sdpa(q[1], dum_k, dum_v, s), atol=1e-12)


def test_two_block_fingerprint():
    # Q = 0: uniform weights over the two blocks -> mean logical block index
    w = S.WORKLOADS["tiny"]
    L, n = w.block_tokens, 5
    j = np.arange(n * L)
    V = np.stack([np.ones(n * L), j // L], axis=1).astype(float)
    K = np.random.default_rng(3).standard_normal((n * L, 2))
    g = geom(w, n)
    sink = O.attend_kind(O.SINK, np.zeros((L, 2)), K, V, g, 1, 1.0, sd_blocks=2)
    dummy = O.attend_kind(O.DUMMY, np.zeros((L, 2)), K, V, g, 1, 1.0, sd_blocks=2)
    np.testing.assert_allclose(sink, np.tile([1, (0 + n - 1) / 2], (L, 1)), atol=1e-12)
    np.testing.assert_allclose(dummy, np.tile([1, (n - 2 + n - 1) / 2], (L, 1)), atol=1e-12)
