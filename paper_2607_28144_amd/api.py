"""Thin torch-facing binding of the C ABI (argument marshalling only).

Every step of the computation runs in the HIP kernels of libregenvc_attn.so;
torch supplies device memory and the current stream.  Tensors are logical
[B, S, H, D] views (any b/s/h strides that are multiples of 8 elements, d
contiguous); LSE tensors are float32 [B, H, Sq].  The scratch memory of the
attention calls (split-tile partials, sized by the call's work plan) is
allocated by torch on the current stream and bound for the call, so the
library itself never allocates on this path.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import List, Optional, Sequence, Tuple

import torch

from . import _lib
from ._lib import RegenvcError  # noqa: F401  (re-export)

_DT = {torch.bfloat16: _lib.BF16, torch.float32: _lib.F32}


def _desc(t: torch.Tensor, name: str, dtype: torch.dtype) -> _lib.Tensor:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor, got {t.device}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.dim() != 4:
        raise ValueError(f"{name} must be [B, S, H, D], got shape {tuple(t.shape)}")
    if t.numel() > 0 and t.shape[3] > 1 and t.stride(3) != 1:
        raise ValueError(f"{name}: the head-dim axis must be contiguous")
    return _lib.Tensor(t.data_ptr(), t.stride(0), t.stride(1), t.stride(2))


def _stream(device: torch.device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _fptr(t: Optional[torch.Tensor], name: str, shape) -> Optional[int]:
    if t is None:
        return None
    if t.dtype != torch.float32 or not t.is_contiguous() or tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must be a contiguous float32 tensor of shape {tuple(shape)}")
    return t.data_ptr()


def _scale(scale: Optional[float], D: int) -> float:
    return float(torch.tensor(1.0 / math.sqrt(D), dtype=torch.float32)) if scale is None else float(scale)


_NEED = {}    # (device index, shape) -> workspace bytes of the call's plan
_N_CU = {}    # device index -> compute units
_TOKEN = {}   # device index -> a 256-byte buffer bound when a call needs no scratch


def _workspace_need(device: torch.device, B, H, Sq, Skv, D, Skv2: int = 0) -> int:
    """Scratch bytes of one attention call (the library's host-only plan query
    with this device's compute-unit count)."""
    idx = device.index if device.index is not None else torch.cuda.current_device()
    # the library picks its kernel, and with it the plan, by this variable too
    key = (idx, B, H, Sq, Skv, Skv2, D, os.environ.get("REGENVC_ATTN_SCHEDULE"))
    need = _NEED.get(key)
    if need is None:
        if idx not in _N_CU:
            _N_CU[idx] = torch.cuda.get_device_properties(idx).multi_processor_count
        if Skv < 1 or B * H * Sq == 0:
            need = 0
        else:
            plan = _lib.AttnPlan()
            lib = _lib.load()
            if Skv2 > 0:
                st = lib.regenvc_cross_attn_dual_plan_query(B, H, Sq, Skv, Skv2, D, _N_CU[idx], ctypes.byref(plan))
            else:
                st = lib.regenvc_attn_plan_query(B, H, Sq, Skv, D, _N_CU[idx], ctypes.byref(plan))
            need = plan.workspace_bytes if st == _lib.OK else 0
        _NEED[key] = need
    return need


def _with_workspace(device: torch.device, need: int, call):
    """Runs call() (one attention entry point) with a torch-allocated scratch
    buffer of `need` bytes bound: the library then allocates nothing.  When
    the call needs none, a small token buffer is bound instead, so that a
    plan mismatch fails loudly rather than falling back to the pool."""
    lib = _lib.load()
    if need > 0:
        buf = torch.empty(need, dtype=torch.uint8, device=device)
    else:
        idx = device.index if device.index is not None else torch.cuda.current_device()
        buf = _TOKEN.get(idx)
        if buf is None:
            buf = _TOKEN[idx] = torch.empty(256, dtype=torch.uint8, device=device)
    _lib.check(lib.regenvc_attn_set_workspace(buf.data_ptr(), need), "regenvc_attn_set_workspace")
    try:
        st = call()
        if st != _lib.OK:  # keep the detail: the unbinding below clears it
            _lib.keep_error_detail()
        return st
    finally:
        lib.regenvc_attn_set_workspace(None, 0)


def pool_draws() -> int:
    """Attention calls in this process that took scratch from the library's
    own pool (regenvc_attn_pool_draws); the calls of this binding never do."""
    return int(_lib.load().regenvc_attn_pool_draws())


def _attn(fn_name: str, q, k, v, scale, out_dtype, out, want_lse, lse_out):
    B, Sq, H, D = q.shape
    Skv = k.shape[1]
    if tuple(k.shape) != (B, Skv, H, D) or tuple(v.shape) != (B, Skv, H, D):
        raise ValueError(f"k/v shapes {tuple(k.shape)}, {tuple(v.shape)} do not match q {tuple(q.shape)}")
    if out is None:
        out = torch.empty((B, Sq, H, D), dtype=out_dtype, device=q.device)
    if lse_out is None and want_lse:
        lse_out = torch.empty((B, H, Sq), dtype=torch.float32, device=q.device)
    qd, kd, vd = _desc(q, "q", torch.bfloat16), _desc(k, "k", torch.bfloat16), _desc(v, "v", torch.bfloat16)
    od = _desc(out, "out", out_dtype)
    lp = _fptr(lse_out, "lse", (B, H, Sq))
    lib = _lib.load()
    need = _workspace_need(q.device, B, H, Sq, Skv, D)
    with torch.cuda.device(q.device):
        if fn_name == "regenvc_attn_partial_fwd":
            st = _with_workspace(q.device, need, lambda: lib.regenvc_attn_partial_fwd(
                ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd), ctypes.byref(od), lp, B, H, Sq, Skv, D,
                _scale(scale, D), _stream(q.device)))
        else:
            st = _with_workspace(q.device, need, lambda: getattr(lib, fn_name)(
                ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd), ctypes.byref(od), _DT[out_dtype], lp, B, H,
                Sq, Skv, D, _scale(scale, D), _stream(q.device)))
    _lib.check(st, fn_name)
    return out, lse_out


def attn_fwd(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, scale: Optional[float] = None,
             out_dtype: torch.dtype = torch.bfloat16, out: Optional[torch.Tensor] = None,
             return_lse: bool = True, lse_out: Optional[torch.Tensor] = None
             ) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """Exact self-attention over all keys (regenvc_attn_fwd).  Returns (O, LSE or None)."""
    return _attn("regenvc_attn_fwd", q, k, v, scale, out_dtype, out, return_lse, lse_out)


def attn_partial_fwd(q: torch.Tensor, k_chunk: torch.Tensor, v_chunk: torch.Tensor,
                     scale: Optional[float] = None, out: Optional[torch.Tensor] = None,
                     lse_out: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Partial attention over one key/value chunk (regenvc_attn_partial_fwd):
    float32 O normalized over the chunk, and its LSE."""
    return _attn("regenvc_attn_partial_fwd", q, k_chunk, v_chunk, scale, torch.float32, out, True, lse_out)


def _chunk_plan(device: torch.device, B, H, Sq, bounds, D) -> int:
    """Scratch bytes of one chunked-partials call (host-only plan query)."""
    idx = device.index if device.index is not None else torch.cuda.current_device()
    key = (idx, B, H, Sq, tuple(bounds), D, os.environ.get("REGENVC_ATTN_SCHEDULE"))
    need = _NEED.get(key)
    if need is None:
        if idx not in _N_CU:
            _N_CU[idx] = torch.cuda.get_device_properties(idx).multi_processor_count
        plan = _lib.AttnPlan()
        arr = (ctypes.c_int32 * len(bounds))(*bounds)
        st = _lib.load().regenvc_attn_partials_plan_query(B, H, Sq, len(bounds) - 1, arr, D, _N_CU[idx],
                                                          ctypes.byref(plan))
        need = _NEED[key] = plan.workspace_bytes if st == _lib.OK else 0
    return need


def attn_partials_fwd(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, bounds: Sequence[int],
                      scale: Optional[float] = None, outs: Optional[Sequence[torch.Tensor]] = None,
                      lse_outs: Optional[Sequence[torch.Tensor]] = None
                      ) -> Tuple[List[torch.Tensor], List[torch.Tensor]]:
    """Partials of every key chunk [bounds[c], bounds[c+1]) in one launch
    (regenvc_attn_partials_fwd): per chunk, float32 O [B, Sq, H, D]
    normalized over the chunk and its LSE [B, H, Sq], as
    attn_partial_fwd gives chunk by chunk."""
    B, Sq, H, D = q.shape
    Skv = k.shape[1]
    if tuple(k.shape) != (B, Skv, H, D) or tuple(v.shape) != (B, Skv, H, D):
        raise ValueError(f"k/v shapes {tuple(k.shape)}, {tuple(v.shape)} do not match q {tuple(q.shape)}")
    n = len(bounds) - 1
    if n < 1:
        raise ValueError("need at least one chunk (two bounds)")
    if outs is None:
        outs = [torch.empty((B, Sq, H, D), dtype=torch.float32, device=q.device) for _ in range(n)]
    if lse_outs is None:
        lse_outs = [torch.empty((B, H, Sq), dtype=torch.float32, device=q.device) for _ in range(n)]
    if len(outs) != n or len(lse_outs) != n:
        raise ValueError(f"{n} chunks need {n} outputs and {n} LSE outputs")
    for t in outs:
        if tuple(t.shape) != (B, Sq, H, D) or t.dtype != torch.float32 or not t.is_contiguous() \
                or t.device != q.device:
            raise ValueError("outs must be contiguous float32 [B, Sq, H, D] tensors on q's device")
    for t in lse_outs:
        if tuple(t.shape) != (B, H, Sq) or t.dtype != torch.float32 or not t.is_contiguous() \
                or t.device != q.device:
            raise ValueError("lse_outs must be contiguous float32 [B, H, Sq] tensors on q's device")
    qd, kd, vd = _desc(q, "q", torch.bfloat16), _desc(k, "k", torch.bfloat16), _desc(v, "v", torch.bfloat16)
    arr = (ctypes.c_int32 * (n + 1))(*[int(x) for x in bounds])
    optrs = (ctypes.c_void_p * n)(*[t.data_ptr() for t in outs])
    lptrs = (ctypes.c_void_p * n)(*[t.data_ptr() for t in lse_outs])
    lib = _lib.load()
    need = _chunk_plan(q.device, B, H, Sq, [int(x) for x in bounds], D)
    with torch.cuda.device(q.device):
        st = _with_workspace(q.device, need, lambda: lib.regenvc_attn_partials_fwd(
            ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd), n, arr, optrs, lptrs, B, H, Sq, Skv, D,
            _scale(scale, D), _stream(q.device)))
    _lib.check(st, "regenvc_attn_partials_fwd")
    return list(outs), list(lse_outs)


def attn_ring_accumulate(q: torch.Tensor, k_chunk: torch.Tensor, v_chunk: torch.Tensor, o_run: torch.Tensor,
                         lse_run: torch.Tensor, scale: Optional[float] = None, out: Optional[torch.Tensor] = None,
                         out_dtype: torch.dtype = torch.float32) -> torch.Tensor:
    """Partial attention over one key/value chunk merged into the running
    state (regenvc_attn_ring_accumulate).  o_run: float32 [B, Sq, H, D]
    normalized output so far (ignored where lse_run is -inf); lse_run:
    float32 [B, H, Sq], updated in place.  With out=None the merged output
    goes back into o_run; otherwise into `out` (out_dtype).  Returns the
    tensor that holds the merged output."""
    B, Sq, H, D = q.shape
    Skv = k_chunk.shape[1]
    if tuple(k_chunk.shape) != (B, Skv, H, D) or tuple(v_chunk.shape) != (B, Skv, H, D):
        raise ValueError(f"k/v shapes {tuple(k_chunk.shape)}, {tuple(v_chunk.shape)} do not match q {tuple(q.shape)}")
    if tuple(o_run.shape) != (B, Sq, H, D):
        raise ValueError(f"o_run shape {tuple(o_run.shape)} does not match q {tuple(q.shape)}")
    qd, kd = _desc(q, "q", torch.bfloat16), _desc(k_chunk, "k_chunk", torch.bfloat16)
    vd, rd = _desc(v_chunk, "v_chunk", torch.bfloat16), _desc(o_run, "o_run", torch.float32)
    lp = _fptr(lse_run, "lse_run", (B, H, Sq))
    if lp is None:
        raise ValueError("lse_run is required")
    if out is None:
        od, dt, res = None, _lib.F32, o_run
    else:
        if tuple(out.shape) != (B, Sq, H, D):
            raise ValueError(f"out shape {tuple(out.shape)} does not match q {tuple(q.shape)}")
        od, dt, res = _desc(out, "out", out_dtype), _DT[out_dtype], out
    lib = _lib.load()
    need = _workspace_need(q.device, B, H, Sq, Skv, D)
    with torch.cuda.device(q.device):
        st = _with_workspace(q.device, need, lambda: lib.regenvc_attn_ring_accumulate(
            ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd), ctypes.byref(rd), lp,
            ctypes.byref(od) if od is not None else None, dt, B, H, Sq, Skv, D, _scale(scale, D),
            _stream(q.device)))
    _lib.check(st, "regenvc_attn_ring_accumulate")
    return res


def cross_attn_fwd(q: torch.Tensor, k_ctx: torch.Tensor, v_ctx: torch.Tensor, scale: Optional[float] = None,
                   out_dtype: torch.dtype = torch.bfloat16, out: Optional[torch.Tensor] = None,
                   return_lse: bool = True, lse_out: Optional[torch.Tensor] = None
                   ) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """Cross-attention to conditioning tokens (regenvc_cross_attn_fwd)."""
    return _attn("regenvc_cross_attn_fwd", q, k_ctx, v_ctx, scale, out_dtype, out, return_lse, lse_out)


def cross_attn_dual_fwd(q: torch.Tensor, k_txt: torch.Tensor, v_txt: torch.Tensor, k_img: torch.Tensor,
                        v_img: torch.Tensor, scale: Optional[float] = None, out: Optional[torch.Tensor] = None,
                        return_lse: bool = True, lse_txt: Optional[torch.Tensor] = None,
                        lse_img: Optional[torch.Tensor] = None):
    """Text and image cross-attention summed, Q read once
    (regenvc_cross_attn_dual_fwd).  Returns (O bf16, LSE_txt, LSE_img) -- the
    LSEs None unless return_lse or given."""
    B, Sq, H, D = q.shape
    St, Si = k_txt.shape[1], k_img.shape[1]
    for name, t, S in [("k_txt", k_txt, St), ("v_txt", v_txt, St), ("k_img", k_img, Si), ("v_img", v_img, Si)]:
        if tuple(t.shape) != (B, S, H, D):
            raise ValueError(f"{name} shape {tuple(t.shape)} does not match q {tuple(q.shape)}")
    if out is None:
        out = torch.empty((B, Sq, H, D), dtype=torch.bfloat16, device=q.device)
    if return_lse:
        lse_txt = lse_txt if lse_txt is not None else torch.empty((B, H, Sq), dtype=torch.float32, device=q.device)
        lse_img = lse_img if lse_img is not None else torch.empty((B, H, Sq), dtype=torch.float32, device=q.device)
    descs = [_desc(t, n, torch.bfloat16) for t, n in
             [(q, "q"), (k_txt, "k_txt"), (v_txt, "v_txt"), (k_img, "k_img"), (v_img, "v_img"), (out, "out")]]
    lt, li = _fptr(lse_txt, "lse_txt", (B, H, Sq)), _fptr(lse_img, "lse_img", (B, H, Sq))
    lib = _lib.load()
    need = _workspace_need(q.device, B, H, Sq, St, D, Skv2=Si)
    with torch.cuda.device(q.device):
        st = _with_workspace(q.device, need, lambda: lib.regenvc_cross_attn_dual_fwd(
            ctypes.byref(descs[0]), ctypes.byref(descs[1]), ctypes.byref(descs[2]), St, ctypes.byref(descs[3]),
            ctypes.byref(descs[4]), Si, ctypes.byref(descs[5]), lt, li, B, H, Sq, D, _scale(scale, D),
            _stream(q.device)))
    _lib.check(st, "regenvc_cross_attn_dual_fwd")
    return out, lse_txt, lse_img


def lse_merge(o_parts: Sequence[torch.Tensor], lse_parts: Sequence[torch.Tensor],
              out_dtype: torch.dtype = torch.bfloat16, out: Optional[torch.Tensor] = None,
              return_lse: bool = True, lse_out: Optional[torch.Tensor] = None
              ) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """Log-sum-exp merge of chunk partials (regenvc_lse_merge)."""
    n = len(o_parts)
    if n != len(lse_parts) or n < 1:
        raise ValueError("need the same, non-zero number of o_parts and lse_parts")
    B, Sq, H, D = o_parts[0].shape
    for t in o_parts:
        if tuple(t.shape) != (B, Sq, H, D) or t.dtype != torch.float32 or not t.is_contiguous() \
                or t.device != o_parts[0].device:
            raise ValueError("o_parts must be contiguous float32 [B, Sq, H, D] tensors on one device")
    for t in lse_parts:
        if tuple(t.shape) != (B, H, Sq) or t.dtype != torch.float32 or not t.is_contiguous() \
                or t.device != o_parts[0].device:
            raise ValueError("lse_parts must be contiguous float32 [B, H, Sq] tensors on one device")
    dev = o_parts[0].device
    if out is None:
        out = torch.empty((B, Sq, H, D), dtype=out_dtype, device=dev)
    if lse_out is None and return_lse:
        lse_out = torch.empty((B, H, Sq), dtype=torch.float32, device=dev)
    od = _desc(out, "out", out_dtype)
    optrs = (ctypes.c_void_p * n)(*[t.data_ptr() for t in o_parts])
    lptrs = (ctypes.c_void_p * n)(*[t.data_ptr() for t in lse_parts])
    lp = _fptr(lse_out, "lse", (B, H, Sq))
    lib = _lib.load()
    with torch.cuda.device(dev):
        st = lib.regenvc_lse_merge(optrs, lptrs, n, ctypes.byref(od), _DT[out_dtype], lp, B, H, Sq, D, _stream(dev))
    _lib.check(st, "regenvc_lse_merge")
    return out, lse_out


def attn_plan(B: int, H: int, Sq: int, Skv: int, D: int, n_cu: int = 256, Skv2: int = 0) -> dict:
    """Work plan of one attention call of this shape on n_cu compute units
    (regenvc_attn_plan_query, or regenvc_cross_attn_dual_plan_query with a
    second context of Skv2 keys; host-only): query/key tile counts, whole and
    split query tiles, key ranges per split tile, workspace bytes."""
    plan = _lib.AttnPlan()
    lib = _lib.load()
    if Skv2:
        st = lib.regenvc_cross_attn_dual_plan_query(B, H, Sq, Skv, Skv2, D, n_cu, ctypes.byref(plan))
        _lib.check(st, "regenvc_cross_attn_dual_plan_query")
    else:
        st = lib.regenvc_attn_plan_query(B, H, Sq, Skv, D, n_cu, ctypes.byref(plan))
        _lib.check(st, "regenvc_attn_plan_query")
    return {f: getattr(plan, f) for f, _ in _lib.AttnPlan._fields_}


def qk_norm_rope(q: torch.Tensor, k: torch.Tensor, w_q: torch.Tensor, w_k: torch.Tensor, grid,
                 token0: int = 0, eps: float = 1e-6, theta: float = 10000.0,
                 q_out: Optional[torch.Tensor] = None, k_out: Optional[torch.Tensor] = None
                 ) -> Tuple[torch.Tensor, torch.Tensor]:
    """q/k RMSNorm over all H*D channels of each token, then 3D rotary
    embedding per head over a (frames, rows, cols) latent grid
    (regenvc_qk_norm_rope).  q, k: bf16 [B, S, H, D]; w_q, w_k: bf16 [H*D]
    contiguous.  Outputs may be q and k themselves (in place).  Returns
    (q_out, k_out)."""
    B, S, H, D = q.shape
    if tuple(k.shape) != (B, S, H, D):
        raise ValueError(f"k shape {tuple(k.shape)} does not match q {tuple(q.shape)}")
    for name, w in (("w_q", w_q), ("w_k", w_k)):
        if not isinstance(w, torch.Tensor) or w.dtype != torch.bfloat16 or w.device != q.device \
                or not w.is_contiguous() or w.numel() != H * D:
            raise ValueError(f"{name} must be a contiguous bf16 device tensor of {H * D} elements")
    q_out = torch.empty_like(q) if q_out is None else q_out
    k_out = torch.empty_like(k) if k_out is None else k_out
    qi, ki = _desc(q, "q", torch.bfloat16), _desc(k, "k", torch.bfloat16)
    qo, ko = _desc(q_out, "q_out", torch.bfloat16), _desc(k_out, "k_out", torch.bfloat16)
    gf, gh, gw = (int(x) for x in grid)
    lib = _lib.load()
    with torch.cuda.device(q.device):
        st = lib.regenvc_qk_norm_rope(ctypes.byref(qi), ctypes.byref(ki), w_q.data_ptr(), w_k.data_ptr(),
                                      ctypes.byref(qo), ctypes.byref(ko), B, S, H, D, gf, gh, gw, int(token0),
                                      float(eps), float(theta), _stream(q.device))
    _lib.check(st, "regenvc_qk_norm_rope")
    return q_out, k_out
