"""Python binding of the HeadCast C ABI (include/headcast.h).

Argument marshalling only: every step of the routed-attention path runs in the
HIP library.  torch supplies device memory (``tensor.data_ptr()``) and the
current stream; nothing here computes.  If the library is missing this module
raises on import instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libheadcast.so")

HC_OK, HC_E_INVAL, HC_E_STATE, HC_E_ORDER, HC_E_NOMEM, HC_E_DEVICE = 0, -1, -2, -3, -4, -5
SINK, DUMMY, SPATIAL, GLOBAL = 0, 1, 2, 3
N_STATS = 6
K_DENSE, K_SPATIAL, K_SCATTER, K_STATS, K_COMBINE = 0, 1, 2, 3, 4
CLS_O_REF, CLS_O_SINK, CLS_O_DUMMY, CLS_O_SPATIAL = 0, 1, 2, 3

EXPORTS = ("hc_config_default", "hc_validate_config", "hc_status_string", "hc_last_error",
           "hc_ring_slot", "hc_create", "hc_destroy", "hc_classify_heads", "hc_classify_outputs",
           "hc_set_head_types",
           "hc_get_layout", "hc_append_block", "hc_attention", "hc_attention_static",
           "hc_memory_bytes", "hc_profile_enable", "hc_profile_read")
STATIC_SCRATCH_BYTES = 64 << 20   # HC_STATIC_SCRATCH_BYTES


class HCConfig(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "n_heads", "head_dim", "grid_h", "grid_w", "frames_per_block",
        "window_blocks", "spatial_radius", "proxy_radius")] + [
        (n, ctypes.c_float) for n in (
            "theta_sink", "theta_dummy", "theta_spatial", "theta_score", "gamma",
            "softmax_scale")] + [("spatial_cell", ctypes.c_int32), ("sd_blocks", ctypes.c_int32)]


class HeadCastError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = status


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"HeadCast library not built: {LIB_PATH} is missing "
                          "(run `python -m paper_2607_20125_amd.build`)")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, U8P, DP = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                            ctypes.POINTER(ctypes.c_uint8), ctypes.POINTER(ctypes.c_double))
    I32P = ctypes.POINTER(ctypes.c_int32)
    CP = ctypes.POINTER(HCConfig)
    sig = {
        "hc_config_default": (None, [CP]),
        "hc_validate_config": (ctypes.c_int, [CP]),
        "hc_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "hc_last_error": (ctypes.c_char_p, [P]),
        "hc_ring_slot": (I32, [I64, I32]),
        "hc_create": (ctypes.c_int, [CP, ctypes.c_int, ctypes.POINTER(P)]),
        "hc_destroy": (None, [P]),
        "hc_classify_heads": (ctypes.c_int, [P, ctypes.c_int, I64, P, P, P, U8P, DP, P]),
        "hc_classify_outputs": (ctypes.c_int, [P, ctypes.c_int, P, P]),
        "hc_set_head_types": (ctypes.c_int, [P, ctypes.c_int, U8P, I64, P, P, P]),
        "hc_get_layout": (ctypes.c_int, [P, ctypes.c_int, I32P, I32P]),
        "hc_append_block": (ctypes.c_int, [P, ctypes.c_int, I64, P, P, P]),
        "hc_attention": (ctypes.c_int, [P, ctypes.c_int, P, U8P, P, P]),
        "hc_attention_static": (ctypes.c_int, [P, ctypes.c_int, P, U8P, P, P]),
        "hc_memory_bytes": (ctypes.c_int, [P, ctypes.POINTER(I64)]),
        "hc_profile_enable": (ctypes.c_int, [P, ctypes.c_int]),
        "hc_profile_read": (ctypes.c_int, [P, ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                           ctypes.POINTER(I64)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype, fn.argtypes = res, args
    return lib


lib = _load()


def status_string(s: int) -> str:
    return lib.hc_status_string(s).decode()


def ring_slot(block: int, window_blocks: int) -> int:
    return lib.hc_ring_slot(block, window_blocks)


def default_config() -> HCConfig:
    c = HCConfig()
    lib.hc_config_default(ctypes.byref(c))
    return c


def make_config(**kw) -> HCConfig:
    c = default_config()
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def config_from_workload(w, n_layers=None, spatial_cell=0, sd_blocks=1) -> HCConfig:
    return make_config(n_layers=w.n_layers if n_layers is None else n_layers,
                       n_heads=w.n_heads, head_dim=w.head_dim, grid_h=w.grid_h,
                       grid_w=w.grid_w, frames_per_block=w.frames_per_block,
                       window_blocks=w.window_blocks, spatial_radius=w.spatial_radius,
                       proxy_radius=w.proxy_radius, spatial_cell=spatial_cell,
                       sd_blocks=sd_blocks)


def validate_config(cfg: HCConfig) -> int:
    return lib.hc_validate_config(ctypes.byref(cfg))


def _u8(types) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(types, dtype=np.uint8))


def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


class Context:
    """Owns one hc_ctx (all layers' compact buffers) on one device."""

    def __init__(self, cfg: HCConfig, device: int = 0):
        self.cfg = cfg
        self._h = ctypes.c_void_p()
        st = lib.hc_create(ctypes.byref(cfg), device, ctypes.byref(self._h))
        if st != HC_OK:
            raise HeadCastError(st, f"hc_create: {status_string(st)}")
        self.L = cfg.frames_per_block * cfg.grid_h * cfg.grid_w

    def close(self):
        if self._h:
            lib.hc_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _check(self, st: int, what: str):
        if st != HC_OK:
            msg = lib.hc_last_error(self._h).decode()
            raise HeadCastError(st, f"{what}: {status_string(st)}: {msg}")

    def _tensor(self, t, dtype_name: str, shape):
        import torch
        dt = {"bf16": torch.bfloat16, "f32": torch.float32}[dtype_name]
        if t.dtype != dt or not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"expected a contiguous {dtype_name} CUDA tensor, got "
                             f"{t.dtype} on {t.device} (contiguous={t.is_contiguous()})")
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"expected shape {tuple(shape)}, got {tuple(t.shape)}")
        return ctypes.c_void_p(t.data_ptr())

    def _win_shape(self, n_blocks):
        c = self.cfg
        return (c.n_heads, n_blocks * self.L, c.head_dim)

    def _blk_shape(self):
        c = self.cfg
        return (c.n_heads, self.L, c.head_dim)

    def set_head_types(self, layer: int, types, cur_block: int, k_win, v_win):
        n = min(cur_block + 1, self.cfg.window_blocks)
        ty = _u8(types)
        self._check(lib.hc_set_head_types(
            self._h, layer, ty.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)), cur_block,
            self._tensor(k_win, "bf16", self._win_shape(n)),
            self._tensor(v_win, "bf16", self._win_shape(n)), _stream()), "hc_set_head_types")

    def classify_heads(self, layer: int, cur_block: int, q, k_win, v_win):
        H = self.cfg.n_heads
        types = np.zeros(H, dtype=np.uint8)
        stats = np.zeros((H, N_STATS), dtype=np.float64)
        W = self.cfg.window_blocks
        self._check(lib.hc_classify_heads(
            self._h, layer, cur_block, self._tensor(q, "bf16", self._blk_shape()),
            self._tensor(k_win, "bf16", self._win_shape(W)),
            self._tensor(v_win, "bf16", self._win_shape(W)),
            types.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)),
            stats.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), _stream()),
            "hc_classify_heads")
        return types, stats

    def classify_outputs(self, which: int, dst):
        """hc_classify_outputs: copy classification output `which` (CLS_O_REF,
        CLS_O_SINK, CLS_O_DUMMY, CLS_O_SPATIAL) of the last classification into
        `dst` (float32 [H][L][d] on the device)."""
        self._check(lib.hc_classify_outputs(self._h, which,
                                            self._tensor(dst, "f32", self._blk_shape()),
                                            _stream()), "hc_classify_outputs")

    def get_layout(self, layer: int):
        H, W = self.cfg.n_heads, self.cfg.window_blocks
        hs = np.zeros(H, dtype=np.int32)
        ring = np.zeros(W, dtype=np.int32)
        I32P = ctypes.POINTER(ctypes.c_int32)
        self._check(lib.hc_get_layout(self._h, layer, hs.ctypes.data_as(I32P),
                                      ring.ctypes.data_as(I32P)), "hc_get_layout")
        return hs, ring

    def append_block(self, layer: int, block: int, k_blk, v_blk):
        self._check(lib.hc_append_block(
            self._h, layer, block, self._tensor(k_blk, "bf16", self._blk_shape()),
            self._tensor(v_blk, "bf16", self._blk_shape()), _stream()), "hc_append_block")

    def attention(self, layer: int, q, types, o):
        ty = _u8(types)
        self._check(lib.hc_attention(
            self._h, layer, self._tensor(q, "bf16", self._blk_shape()),
            ty.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)),
            self._tensor(o, "f32", self._blk_shape()), _stream()), "hc_attention")

    def attention_static(self, layer: int, q, types, o):
        """hc_attention_static: the same layer-step in the library's fixed
        device scratch (no device allocation)."""
        ty = _u8(types)
        self._check(lib.hc_attention_static(
            self._h, layer, self._tensor(q, "bf16", self._blk_shape()),
            ty.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)),
            self._tensor(o, "f32", self._blk_shape()), _stream()), "hc_attention_static")

    def memory_bytes(self) -> int:
        b = ctypes.c_int64()
        self._check(lib.hc_memory_bytes(self._h, ctypes.byref(b)), "hc_memory_bytes")
        return b.value

    def profile_enable(self, on: bool = True):
        self._check(lib.hc_profile_enable(self._h, 1 if on else 0), "hc_profile_enable")

    def profile_read(self, kind: int):
        ms, n = ctypes.c_double(), ctypes.c_int64()
        self._check(lib.hc_profile_read(self._h, kind, ctypes.byref(ms), ctypes.byref(n)),
                    "hc_profile_read")
        return ms.value, n.value
