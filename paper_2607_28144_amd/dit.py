"""Thin torch-facing binding of the diffusion-transformer block kernels
(include/regenvc_dit.h): argument marshalling only; every step runs in the
HIP kernels of libregenvc_attn.so on torch's current stream.

Tensors: activations are bf16 or (the residual stream) float32 [rows, C]
with unit column stride; linear weights bf16 [out, in] contiguous; biases
and normalization scales bf16 [n]; modulation vectors float32.
"""
from __future__ import annotations

import ctypes
from typing import Dict, Optional

import torch

from . import _lib

EPI = {"bias": 0, "bias_gelu": 1, "gated_residual": 2}


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _rows(t: torch.Tensor, name: str, dtype: torch.dtype) -> int:
    if t.device.type != "cuda" or t.dtype != dtype or t.dim() != 2 or (t.shape[1] > 1 and t.stride(1) != 1):
        raise ValueError(f"{name} must be a {dtype} device tensor [rows, cols] with unit column stride")
    return t.stride(0)


def _vec(t: Optional[torch.Tensor], name: str, dtype: torch.dtype, n: int) -> Optional[int]:
    if t is None:
        return None
    if t.device.type != "cuda" or t.dtype != dtype or not t.is_contiguous() or t.numel() != n:
        raise ValueError(f"{name} must be a contiguous {dtype} device tensor of {n} elements")
    return t.data_ptr()


def linear_fwd(a: torch.Tensor, w: torch.Tensor, bias: Optional[torch.Tensor] = None, epilogue: str = "bias",
               gate: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """y = a w^T (+ bias) with a fused epilogue (regenvc_linear_fwd):
    'bias' -> bf16 out, 'bias_gelu' -> bf16 gelu_tanh(y), 'gated_residual' ->
    out (float32, required) += gate * y."""
    M, K = a.shape
    N = w.shape[0]
    lda = _rows(a, "a", torch.bfloat16)
    if tuple(w.shape) != (N, K) or not w.is_contiguous() or w.dtype != torch.bfloat16:
        raise ValueError("w must be a contiguous bf16 [N, K] tensor")
    epi = EPI[epilogue]
    if out is None:
        if epi == 2:
            raise ValueError("the gated-residual epilogue needs out (the float32 residual stream)")
        out = torch.empty((M, N), dtype=torch.bfloat16, device=a.device)
    ldo = _rows(out, "out", torch.float32 if epi == 2 else torch.bfloat16)
    st = _lib.load().regenvc_linear_fwd(a.data_ptr(), lda, w.data_ptr(), _vec(bias, "bias", torch.bfloat16, N),
                                        _vec(gate, "gate", torch.float32, N), out.data_ptr(), ldo, M, N, K, epi,
                                        _stream(a.device))
    _lib.check(st, "regenvc_linear_fwd")
    return out


def layer_norm_fwd(x: torch.Tensor, shift=None, scale=None, w=None, b=None, eps: float = 1e-6,
                   out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """bf16 LN(x)(1 + scale) + shift (float32 shift/scale), or LN(x) w + b
    (bf16 w, b), of float32 rows x (regenvc_layer_norm_fwd)."""
    rows, C = x.shape
    ldx = _rows(x, "x", torch.float32)
    out = torch.empty((rows, C), dtype=torch.bfloat16, device=x.device) if out is None else out
    ldy = _rows(out, "out", torch.bfloat16)
    st = _lib.load().regenvc_layer_norm_fwd(
        x.data_ptr(), ldx, out.data_ptr(), ldy, _vec(shift, "shift", torch.float32, C),
        _vec(scale, "scale", torch.float32, C), _vec(w, "w", torch.bfloat16, C), _vec(b, "b", torch.bfloat16, C),
        rows, C, float(eps), _stream(x.device))
    _lib.check(st, "regenvc_layer_norm_fwd")
    return out


def rms_norm_fwd(x: torch.Tensor, w: torch.Tensor, eps: float = 1e-6,
                 out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """bf16 x / rms(x) w of bf16 rows (regenvc_rms_norm_fwd); out may be x."""
    rows, C = x.shape
    ldx = _rows(x, "x", torch.bfloat16)
    out = torch.empty_like(x) if out is None else out
    ldy = _rows(out, "out", torch.bfloat16)
    st = _lib.load().regenvc_rms_norm_fwd(x.data_ptr(), ldx, out.data_ptr(), ldy, _vec(w, "w", torch.bfloat16, C),
                                          rows, C, float(eps), _stream(x.device))
    _lib.check(st, "regenvc_rms_norm_fwd")
    return out


def modulation(w_mod: torch.Tensor, b_mod: torch.Tensor, e: torch.Tensor,
               out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """float32 W_mod silu(e) + b_mod (regenvc_dit_modulation)."""
    rows, C = w_mod.shape
    out = torch.empty(rows, dtype=torch.float32, device=e.device) if out is None else out
    st = _lib.load().regenvc_dit_modulation(_vec(w_mod, "w_mod", torch.bfloat16, rows * C),
                                            _vec(b_mod, "b_mod", torch.bfloat16, rows),
                                            _vec(e, "e", torch.float32, C), _vec(out, "out", torch.float32, rows),
                                            rows, C, _stream(e.device))
    _lib.check(st, "regenvc_dit_modulation")
    return out


class DitBlock:
    """One diffusion-transformer block on the GPU: its bf16 parameters
    (device tensors, names as in regenvc_dit_params) and a workspace sized
    per shape, allocated by torch.  forward() runs regenvc_dit_block_fwd,
    updating the float32 residual stream in place."""

    def __init__(self, params: Dict[str, torch.Tensor], heads: int = 12):
        missing = [n for n in _lib.DIT_PARAM_NAMES if n not in params]
        if missing:
            raise ValueError(f"missing parameters: {missing}")
        self.params = params
        self.C = params["w_o"].shape[0]
        self.F = params["w_1"].shape[0]
        self.heads = heads
        for n in _lib.DIT_PARAM_NAMES:
            t = params[n]
            if t.dtype != torch.bfloat16 or t.device.type != "cuda" or not t.is_contiguous():
                raise ValueError(f"parameter {n} must be a contiguous bf16 device tensor")
        self._c = _lib.DitParams(*[params[n].data_ptr() for n in _lib.DIT_PARAM_NAMES])
        self._ws = {}

    def workspace_bytes(self, S: int, S_ctx: int, device) -> int:
        n_cu = torch.cuda.get_device_properties(device).multi_processor_count
        out = ctypes.c_int64()
        st = _lib.load().regenvc_dit_block_workspace(S, S_ctx, self.C, self.heads, self.F, n_cu, ctypes.byref(out))
        _lib.check(st, "regenvc_dit_block_workspace")
        return out.value

    def forward(self, x: torch.Tensor, e: torch.Tensor, ctx_k: torch.Tensor, ctx_v: torch.Tensor, grid,
                token0: int = 0) -> torch.Tensor:
        """x: float32 [S, C] contiguous (updated in place); e: float32 [C];
        ctx_k, ctx_v: bf16 [S_ctx, heads, D] contiguous; grid = (frames,
        rows, cols) of the latent window."""
        S, C = x.shape
        S_ctx = ctx_k.shape[0]
        if C != self.C or x.dtype != torch.float32 or not x.is_contiguous():
            raise ValueError(f"x must be a contiguous float32 [S, {self.C}] tensor")
        for name, t in (("ctx_k", ctx_k), ("ctx_v", ctx_v)):
            if t.dtype != torch.bfloat16 or not t.is_contiguous() or t.numel() != S_ctx * C:
                raise ValueError(f"{name} must be a contiguous bf16 [S_ctx, heads, D] tensor")
        key = (x.device.index, S, S_ctx)
        if key not in self._ws:
            self._ws[key] = torch.empty(self.workspace_bytes(S, S_ctx, x.device), dtype=torch.uint8,
                                        device=x.device)
        ws = self._ws[key]
        gf, gh, gw = (int(v) for v in grid)
        st = _lib.load().regenvc_dit_block_fwd(
            x.data_ptr(), _vec(e, "e", torch.float32, C), ctypes.byref(self._c), ctx_k.data_ptr(), ctx_v.data_ptr(),
            S_ctx, S, C, self.heads, self.F, gf, gh, gw, int(token0), ws.data_ptr(), ws.numel(), _stream(x.device))
        _lib.check(st, "regenvc_dit_block_fwd")
        return x
