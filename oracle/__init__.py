"""Reference oracle -- TEST INFRASTRUCTURE ONLY.

Plain fp64 CPU definitions of what the GPU path computes (see oracle.c for
the formulas and the paper passages they follow).  Only the tests, the smoke
check and the benchmark's CPU-baseline leg may use this package; the product
library neither imports nor links it, and it imports nothing from the
product.  Inputs are bf16 bit patterns (uint16 numpy arrays, logical
[B, S, H, D], any strides); outputs are float64.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

ORACLE_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(ORACLE_DIR, "liboracle.so")
_lib = None


def open_library(path: str) -> ctypes.CDLL:
    """Loads an oracle shared library and declares its functions."""
    lib = ctypes.CDLL(path)
    p, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    lib.oracle_attn.argtypes = [p, i64, i64, i64, p, i64, i64, i64, p, i64, i64, i64, p, p,
                                i32, i32, i32, i32, i32, ctypes.c_float]
    lib.oracle_attn.restype = i32
    lib.oracle_merge.argtypes = [ctypes.POINTER(p), ctypes.POINTER(p), i32, p, p, i32, i32, i32, i32]
    lib.oracle_merge.restype = i32
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = i32
    lib.oracle_set_num_threads.argtypes = [i32]
    lib.oracle_set_num_threads.restype = None
    lib.oracle_norm_rope.argtypes = [p, i64, i64, i64, p, p, i32, i32, i32, i32, i32, i32, i32, i32,
                                     ctypes.c_float, ctypes.c_float]
    lib.oracle_norm_rope.restype = i32
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            from .build import build
            build()
        _lib = open_library(LIB_PATH)
    return _lib


def _strides(a: np.ndarray):
    if a.dtype != np.uint16 or a.ndim != 4:
        raise TypeError("expected a uint16 (bf16 bits) array of shape [B, S, H, D]")
    if a.strides[3] != 2:
        raise ValueError("the head-dim axis must be contiguous")
    return tuple(s // 2 for s in a.strides[:3])


def attn(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float, lib=None):
    """Exact attention of every query over all keys of k/v.
    Returns (O float64 [B,Sq,H,D], LSE float64 [B,H,Sq]).  A key/value chunk's
    partial result is this function applied to the chunk's rows."""
    B, Sq, H, D = q.shape
    Skv = k.shape[1]
    assert k.shape == (B, Skv, H, D) and v.shape == (B, Skv, H, D)
    o = np.empty((B, Sq, H, D), dtype=np.float64)
    lse = np.empty((B, H, Sq), dtype=np.float64)
    lib = lib or _load()
    rc = lib.oracle_attn(q.ctypes.data, *_strides(q), k.ctypes.data, *_strides(k), v.ctypes.data, *_strides(v),
                         o.ctypes.data, lse.ctypes.data, B, H, Sq, Skv, D, ctypes.c_float(scale))
    if rc != 0:
        raise ValueError("oracle_attn rejected its arguments")
    return o, lse


def merge(o_parts, lse_parts, lib=None):
    """Log-sum-exp merge of partials over disjoint key chunks (float64 in/out)."""
    n = len(o_parts)
    o_parts = [np.ascontiguousarray(x, dtype=np.float64) for x in o_parts]
    lse_parts = [np.ascontiguousarray(x, dtype=np.float64) for x in lse_parts]
    B, Sq, H, D = o_parts[0].shape
    o = np.empty((B, Sq, H, D), dtype=np.float64)
    lse = np.empty((B, H, Sq), dtype=np.float64)
    optr = (ctypes.c_void_p * n)(*[x.ctypes.data for x in o_parts])
    lptr = (ctypes.c_void_p * n)(*[x.ctypes.data for x in lse_parts])
    rc = (lib or _load()).oracle_merge(optr, lptr, n, o.ctypes.data, lse.ctypes.data, B, H, Sq, D)
    if rc != 0:
        raise ValueError("oracle_merge rejected its arguments")
    return o, lse


def ring_accumulate(o_run, lse_run, q, k, v, scale: float, lib=None):
    """One ring step (paper Sec. 3.5: key/value blocks folded into a running
    result with running-max rescaling): the attention of q over this key/value chunk, merged into the
    running state (o_run, lse_run) of the chunks seen so far by the same
    log-sum-exp identity as merge().  Rows whose lse_run is -inf have seen no
    key; their o_run is not used.  Returns the new (O, LSE), float64."""
    o_c, l_c = attn(q, k, v, scale, lib)
    lse_run = np.asarray(lse_run, dtype=np.float64)
    fresh = np.isneginf(lse_run)                        # [B, H, Sq]
    o_run = np.array(o_run, dtype=np.float64)
    o_run[np.transpose(fresh, (0, 2, 1))] = 0.0         # [B, Sq, H] rows
    return merge([o_run, o_c], [lse_run, l_c], lib)


def cross_attn_dual(q, k_txt, v_txt, k_img, v_img, scale: float, lib=None):
    """Text and image cross-attention summed (paper Sec. 3.9: the video tokens
    are conditioned on both the T5 text and the CLIP image key/values): each
    context has its own softmax, and the two outputs are added.  Returns
    (O float64 [B,Sq,H,D], LSE_txt, LSE_img float64 [B,H,Sq])."""
    o_t, l_t = attn(q, k_txt, v_txt, scale, lib)
    o_i, l_i = attn(q, k_img, v_img, scale, lib)
    return o_t + o_i, l_t, l_i


def norm_rope(x: np.ndarray, w: np.ndarray, grid, token0: int = 0, eps: float = 1e-6, theta: float = 10000.0,
              lib=None):
    """q or k RMSNorm over all H*D channels of a token, then 3D rotary
    embedding per head (see oracle_norm_rope in oracle.c).  x: bf16 bits
    [B, S, H, D]; w: bf16 bits [H*D]; grid = (frames, rows, cols).  Returns
    float64 [B, S, H, D]."""
    B, S, H, D = x.shape
    w = np.ascontiguousarray(w, dtype=np.uint16)
    assert w.shape == (H * D,)
    y = np.empty((B, S, H, D), dtype=np.float64)
    rc = (lib or _load()).oracle_norm_rope(x.ctypes.data, *_strides(x), w.ctypes.data, y.ctypes.data, B, S, H, D,
                                           int(grid[0]), int(grid[1]), int(grid[2]), int(token0),
                                           ctypes.c_float(eps), ctypes.c_float(theta))
    if rc != 0:
        raise ValueError("oracle_norm_rope rejected its arguments")
    return y


def num_threads() -> int:
    return _load().oracle_num_threads()


def set_num_threads(n: int) -> None:
    """Threads of later oracle calls (e.g. 1 to time it on one core)."""
    _load().oracle_set_num_threads(int(n))
