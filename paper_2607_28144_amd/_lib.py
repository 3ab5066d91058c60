"""ctypes declarations of the C ABI in include/regenvc_attn.h."""
from __future__ import annotations

import ctypes
import os
import threading

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libregenvc_attn.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_HIP = 0, 1, 2, 3
BF16, F32 = 0, 1
MAX_PARTS = 16


class Tensor(ctypes.Structure):
    """regenvc_tensor: base pointer + element strides of the b, s, h axes."""
    _fields_ = [("ptr", ctypes.c_void_p), ("stride_b", ctypes.c_int64),
                ("stride_s", ctypes.c_int64), ("stride_h", ctypes.c_int64)]


class AttnPlan(ctypes.Structure):
    """regenvc_attn_plan: the work decomposition of one attention call."""
    _fields_ = [("query_tiles", ctypes.c_int32), ("key_tiles", ctypes.c_int32),
                ("whole_tiles", ctypes.c_int32), ("split_tiles", ctypes.c_int32),
                ("key_ranges", ctypes.c_int32), ("workspace_bytes", ctypes.c_int64),
                ("tile_rows", ctypes.c_int32)]


class VaeTile(ctypes.Structure):
    """regenvc_vae_tile: a tile's core and region (half-open row/column ranges)."""
    _fields_ = [(n, ctypes.c_int32) for n in ("core_y0", "core_y1", "core_x0", "core_x1",
                                              "reg_y0", "reg_y1", "reg_x0", "reg_x1")]


DIT_PARAM_NAMES = ("w_mod", "b_mod", "w_qkv", "b_qkv", "w_qn", "w_kn", "w_o", "b_o", "w_n3", "b_n3", "w_qc",
                   "b_qc", "w_qcn", "w_oc", "b_oc", "w_1", "b_1", "w_2", "b_2")


class DitParams(ctypes.Structure):
    """regenvc_dit_params: device pointers of one block's bf16 parameters."""
    _fields_ = [(n, ctypes.c_void_p) for n in DIT_PARAM_NAMES]


class RegenvcError(RuntimeError):
    def __init__(self, status: int, fn: str, detail: str):
        self.status = status
        super().__init__(f"{fn} failed with status {status}: {detail}")


_PT = ctypes.POINTER(Tensor)
_i32 = ctypes.c_int32
_FP = ctypes.POINTER(ctypes.c_float)
_SIGNATURES = {
    "regenvc_attn_fwd": [_PT, _PT, _PT, _PT, ctypes.c_int, ctypes.c_void_p,
                         _i32, _i32, _i32, _i32, _i32, ctypes.c_float, ctypes.c_void_p],
    "regenvc_attn_fwd_noalloc": [_PT, _PT, _PT, _PT, ctypes.c_int, ctypes.c_void_p,
                                 _i32, _i32, _i32, _i32, _i32, ctypes.c_float, ctypes.c_void_p],
    "regenvc_attn_partial_fwd": [_PT, _PT, _PT, _PT, ctypes.c_void_p,
                                 _i32, _i32, _i32, _i32, _i32, ctypes.c_float, ctypes.c_void_p],
    "regenvc_attn_partials_fwd": [_PT, _PT, _PT, _i32, ctypes.POINTER(_i32), ctypes.POINTER(ctypes.c_void_p),
                                  ctypes.POINTER(ctypes.c_void_p), _i32, _i32, _i32, _i32, _i32, ctypes.c_float,
                                  ctypes.c_void_p],
    "regenvc_attn_partials_plan_query": [_i32, _i32, _i32, _i32, ctypes.POINTER(_i32), _i32, _i32,
                                         ctypes.POINTER(AttnPlan)],
    "regenvc_lse_merge": [ctypes.POINTER(ctypes.c_void_p), ctypes.POINTER(ctypes.c_void_p), _i32,
                          _PT, ctypes.c_int, ctypes.c_void_p, _i32, _i32, _i32, _i32, ctypes.c_void_p],
    "regenvc_attn_ring_accumulate": [_PT, _PT, _PT, _PT, ctypes.c_void_p, _PT, ctypes.c_int,
                                     _i32, _i32, _i32, _i32, _i32, ctypes.c_float, ctypes.c_void_p],
    "regenvc_cross_attn_dual_fwd": [_PT, _PT, _PT, _i32, _PT, _PT, _i32, _PT, ctypes.c_void_p, ctypes.c_void_p,
                                    _i32, _i32, _i32, _i32, ctypes.c_float, ctypes.c_void_p],
    "regenvc_cross_attn_fwd": [_PT, _PT, _PT, _PT, ctypes.c_int, ctypes.c_void_p,
                               _i32, _i32, _i32, _i32, _i32, ctypes.c_float, ctypes.c_void_p],
    "regenvc_attn_plan_query": [_i32, _i32, _i32, _i32, _i32, _i32, ctypes.POINTER(AttnPlan)],
    "regenvc_cross_attn_dual_plan_query": [_i32, _i32, _i32, _i32, _i32, _i32, _i32, ctypes.POINTER(AttnPlan)],
    "regenvc_attn_set_workspace": [ctypes.c_void_p, ctypes.c_int64],
    "regenvc_linear_fwd": [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                           ctypes.c_void_p, ctypes.c_int64, _i32, _i32, _i32, _i32, ctypes.c_void_p],
    "regenvc_layer_norm_fwd": [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                               ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, _i32, _i32, ctypes.c_float,
                               ctypes.c_void_p],
    "regenvc_rms_norm_fwd": [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                             _i32, _i32, ctypes.c_float, ctypes.c_void_p],
    "regenvc_dit_modulation": [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, _i32, _i32,
                               ctypes.c_void_p],
    "regenvc_vae_split": [_i32, _i32, _i32, _i32, _i32, ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32),
                          ctypes.POINTER(ctypes.c_int32)],
    "regenvc_vae_conv3d_fwd": [ctypes.c_void_p, _i32, ctypes.c_void_p, ctypes.c_void_p, _i32, ctypes.c_void_p,
                               _i32, _i32, _i32, _i32, _i32, ctypes.c_void_p, _i32, _i32, _i32, ctypes.c_void_p,
                               ctypes.c_int64, ctypes.c_void_p],
    "regenvc_vae_conv3d_workspace": [_i32, _i32, _i32, _i32, _i32, _i32, _i32, ctypes.POINTER(ctypes.c_int64)],
    "regenvc_vae_blend": [ctypes.c_void_p, ctypes.c_void_p, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32,
                          ctypes.c_void_p, ctypes.c_void_p],
    "regenvc_dit_block_workspace": [_i32, _i32, _i32, _i32, _i32, _i32, ctypes.POINTER(ctypes.c_int64)],
    "regenvc_dit_block_fwd": [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                              _i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32, ctypes.c_void_p,
                              ctypes.c_int64, ctypes.c_void_p],
    "regenvc_qk_norm_rope": [_PT, _PT, ctypes.c_void_p, ctypes.c_void_p, _PT, _PT, _i32, _i32, _i32, _i32,
                             _i32, _i32, _i32, _i32, ctypes.c_float, ctypes.c_float, ctypes.c_void_p],
}

_lib = None


def load(path: str | None = None) -> ctypes.CDLL:
    """Loads the built library (once).  Fails loudly if it has not been built:
    there is no fallback implementation."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise ImportError(f"{p} is missing; build it with `python -m paper_2607_28144_amd.build`")
    lib = ctypes.CDLL(p)
    for name, argtypes in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.argtypes = argtypes
        fn.restype = ctypes.c_int
    lib.regenvc_status_str.argtypes = [ctypes.c_int]
    lib.regenvc_status_str.restype = ctypes.c_char_p
    lib.regenvc_last_error.argtypes = []
    lib.regenvc_last_error.restype = ctypes.c_char_p
    lib.regenvc_attn_pool_draws.argtypes = []
    lib.regenvc_attn_pool_draws.restype = ctypes.c_int64
    if path is None:
        _lib = lib
    return lib


_kept = threading.local()


def keep_error_detail() -> None:
    """Saves the library's error text of the failed call just made on this
    thread, for the next check() (a later successful call clears the text)."""
    _kept.detail = load().regenvc_last_error().decode(errors="replace")


def check(status: int, fn: str) -> None:
    kept = getattr(_kept, "detail", None)
    _kept.detail = None
    if status != OK:
        detail = kept if kept is not None else load().regenvc_last_error().decode(errors="replace")
        raise RegenvcError(status, fn, detail)
