"""The benchmark's work counters against the oracle's brute-force key-set sizes
and the closed forms of the 720P workload."""
import numpy as np
import pytest

from oracle import headcast_oracle as O
from paper_2607_20125_amd import costs as C


@pytest.mark.parametrize("geom", [(8, 8, 2, 4, 1), (5, 7, 3, 2, 2), (6, 9, 1, 3, 4), (30, 52, 3, 7, 4)])
def test_pairs_match_oracle(geom):
    Hg, Wg, F, n, r = geom
    for kind in range(4):
        assert C.pairs(kind, Hg, Wg, F, n, r) == O.in_set_pairs(kind, Hg, Wg, F, n, r)


def test_pairs_match_brute_force_key_sets():
    g = O.Geometry(5, 7, 3, 2)
    for kind in range(4):
        brute = sum(O.key_set(kind, g, t, 2).size for t in range(g.L))
        assert C.pairs(kind, 5, 7, 3, 2, 2) == brute


def test_720p_layer_numbers():
    # per-head GFLOP at 720P: Global 418.04, Sink = Dummy 59.72, Spatial 8.69
    assert C.head_flops(C.GLOBAL, 45, 80, 3, 7, 4, 128) / 1e9 == pytest.approx(418.04, abs=0.01)
    assert C.head_flops(C.SINK, 45, 80, 3, 7, 4, 128) / 1e9 == pytest.approx(59.72, abs=0.01)
    assert C.head_flops(C.SPATIAL, 45, 80, 3, 7, 4, 128) / 1e9 == pytest.approx(8.69, abs=0.01)
    # Spatial compulsory bytes: Q 2.76 MB + K,V 38.7 MB + O 5.5 MB
    assert C.head_bytes(C.SPATIAL, 45, 80, 3, 7, 128) == 10800 * 256 + 2 * 75600 * 256 + 10800 * 512


def test_layer_sums():
    types = np.array([0, 1, 2, 3, 3])
    f = C.layer_flops(types, 8, 8, 2, 4, 1, 64)
    assert f == O.algorithmic_flops(types, 8, 8, 2, 4, 1, 64)
    assert C.layer_flops(types, 8, 8, 2, 4, 1, 64, kinds=(3,)) == 2 * 4 * 64 * 128 * 512


def test_cell_pairs_match_oracle_key_sets():
    # brute force over the oracle's cell key sets on small ragged grids
    from oracle import headcast_oracle as O
    for gh, gw, F, n, c in [(5, 8, 1, 3, 2), (7, 9, 2, 2, 3), (8, 8, 2, 4, 3), (6, 11, 3, 2, 4)]:
        g = O.Geometry(gh, gw, F, n)
        brute = sum(O.keys_spatial_cell(g, t, c).size for t in range(F * gh * gw))
        assert C.cell_pairs(gh, gw, F, n, c) == brute
        assert C.head_flops(C.SPATIAL, gh, gw, F, n, 0, 64, cell=c) == 4 * 64 * brute


def test_cell_sizes_hand_values():
    assert C.cell_sizes(45, 10) == [10, 10, 10, 10, 5]
    assert C.cell_sizes(52, 10) == [10, 10, 10, 10, 12]
    assert C.cell_sizes(30, 10) == [10, 10, 10]
    assert C.cell_sizes(4, 10) == [4]


def test_two_block_pairs_match_oracle_key_sets():
    from oracle import headcast_oracle as O
    for n in (1, 2, 4):
        g = O.Geometry(4, 6, 2, n)
        for kind, fn in ((C.SINK, O.keys_sink), (C.DUMMY, O.keys_dummy)):
            brute = g.L * fn(g, 0, 2).size
            assert C.pairs(kind, 4, 6, 2, n, 0, sd_blocks=2) == brute
