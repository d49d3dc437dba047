"""Host-side checks of the C ABI: the library loads, exports every symbol the
header declares, and its pure host logic (config validation, ring slots,
status strings) behaves as documented.  No compute call needs a GPU here."""
import ctypes
import math
import os
import re

import pytest

from oracle import headcast_oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "headcast.h")


@pytest.fixture(scope="module")
def hcb():
    from paper_2607_20125_amd import headcast
    return headcast


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hc_[a-z_]+)\s*\(", text)))


def test_header_declares_expected_entry_points():
    names = declared_functions()
    for must in ("hc_classify_heads", "hc_append_block", "hc_attention", "hc_set_head_types",
                 "hc_get_layout", "hc_create", "hc_destroy"):
        assert must in names


def test_library_exports_every_declared_symbol(hcb):
    lib = ctypes.CDLL(hcb.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), f"{name} declared in headcast.h but not exported"
    assert sorted(hcb.EXPORTS) == declared_functions()


def test_ring_slot_matches_oracle_simulation(hcb):
    for W in (2, 3, 4, 7, 8):
        for blocks in range(1, 5 * W):
            held = O.simulate_ring(blocks, W)
            for b, slot in held.items():
                assert hcb.ring_slot(b, W) == slot
    assert hcb.ring_slot(-1, 7) == -1
    assert hcb.ring_slot(3, 1) == -1


def test_default_config_is_the_papers(hcb):
    c = hcb.default_config()
    assert (c.n_layers, c.n_heads, c.head_dim, c.frames_per_block, c.window_blocks) == (30, 12, 128, 3, 7)
    assert (c.grid_h, c.grid_w, c.spatial_radius, c.proxy_radius) == (30, 52, 4, 2)
    assert c.theta_sink == c.theta_dummy == c.theta_spatial == pytest.approx(0.95)
    assert c.theta_score == pytest.approx(0.755)
    assert c.gamma == 5.0 and c.softmax_scale == 0.0
    assert c.spatial_cell == 0 and c.sd_blocks == 1
    assert hcb.validate_config(c) == hcb.HC_OK


@pytest.mark.parametrize("field,value", [
    ("head_dim", 96), ("head_dim", 256), ("n_heads", 0), ("n_heads", 65), ("n_layers", 0),
    ("frames_per_block", 0), ("frames_per_block", 5), ("window_blocks", 1),
    ("window_blocks", 33), ("spatial_radius", -1), ("spatial_radius", 13),
    ("proxy_radius", 13), ("grid_w", 0), ("softmax_scale", -1.0),
    ("softmax_scale", float("nan")), ("gamma", float("inf")),
    ("spatial_cell", 1), ("spatial_cell", 65), ("spatial_cell", -2),
    ("sd_blocks", 0), ("sd_blocks", 3),
])
def test_validate_config_rejects(hcb, field, value):
    c = hcb.default_config()
    setattr(c, field, value)
    assert hcb.validate_config(c) == hcb.HC_E_INVAL


def test_validate_config_two_block_needs_previous_block_in_window(hcb):
    c = hcb.make_config(sd_blocks=2, window_blocks=2)
    assert hcb.validate_config(c) == hcb.HC_E_INVAL
    c = hcb.make_config(sd_blocks=2, window_blocks=3)
    assert hcb.validate_config(c) == hcb.HC_OK


def test_validate_config_block_multiple_of_8(hcb):
    c = hcb.make_config(grid_h=3, grid_w=5, frames_per_block=1)      # L = 15
    assert hcb.validate_config(c) == hcb.HC_E_INVAL
    c = hcb.make_config(grid_h=3, grid_w=8, frames_per_block=1)      # L = 24
    assert hcb.validate_config(c) == hcb.HC_OK


def test_create_rejects_bad_config_before_touching_a_device(hcb):
    c = hcb.default_config()
    c.head_dim = 100
    h = ctypes.c_void_p()
    assert hcb.lib.hc_create(ctypes.byref(c), 0, ctypes.byref(h)) == hcb.HC_E_INVAL
    assert not h.value
    assert hcb.lib.hc_create(ctypes.byref(hcb.default_config()), 0, None) == hcb.HC_E_INVAL


def test_create_without_gpu_reports_device_error(hcb):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    h = ctypes.c_void_p()
    st = hcb.lib.hc_create(ctypes.byref(hcb.default_config()), 0, ctypes.byref(h))
    assert st == hcb.HC_E_DEVICE and not h.value


def test_null_context_calls_are_rejected(hcb):
    L = hcb.lib
    assert L.hc_attention(None, 0, None, None, None, None) == hcb.HC_E_INVAL
    assert L.hc_attention_static(None, 0, None, None, None, None) == hcb.HC_E_INVAL
    assert L.hc_classify_outputs(None, hcb.CLS_O_REF, None, None) == hcb.HC_E_INVAL
    assert L.hc_append_block(None, 0, 0, None, None, None) == hcb.HC_E_INVAL
    assert L.hc_get_layout(None, 0, None, None) == hcb.HC_E_INVAL
    assert L.hc_profile_enable(None, 1) == hcb.HC_E_INVAL
    assert L.hc_last_error(None) == b""
    L.hc_destroy(None)


def test_status_strings(hcb):
    for s in (0, -1, -2, -3, -4, -5):
        assert hcb.status_string(s)
    assert hcb.status_string(-99) == "unknown status"


def test_validate_config_spatial_cells(hcb):
    # the paper's 10 x 10 cells at every Wan-shaped grid; at most 64 cells per axis
    for gh, gw in [(30, 52), (45, 80), (68, 120)]:
        assert hcb.validate_config(hcb.make_config(grid_h=gh, grid_w=gw, spatial_cell=10)) == hcb.HC_OK
    assert hcb.validate_config(hcb.make_config(grid_h=8, grid_w=8, spatial_cell=3)) == hcb.HC_OK
    c = hcb.make_config(grid_h=8, grid_w=272, frames_per_block=1, spatial_cell=4)   # 68 cells
    assert hcb.validate_config(c) == hcb.HC_E_INVAL
    c.spatial_cell = 5                                                             # 54 cells
    assert hcb.validate_config(c) == hcb.HC_OK


def test_classify_output_ids_match_header(hcb):
    text = open(HEADER).read()
    for name in ("REF", "SINK", "DUMMY", "SPATIAL"):
        m = re.search(rf"HC_CLS_O_{name}\s*=\s*(\d+)", text)
        assert m and int(m.group(1)) == getattr(hcb, f"CLS_O_{name}")


def test_static_scratch_size_matches_header(hcb):
    text = open(HEADER).read()
    m = re.search(r"#define HC_STATIC_SCRATCH_BYTES \((\d+)u << (\d+)\)", text)
    assert m, "HC_STATIC_SCRATCH_BYTES not found"
    assert int(m.group(1)) << int(m.group(2)) == hcb.STATIC_SCRATCH_BYTES
