"""Thin torch-facing binding of the spatially split VAE tile kernels
(include/regenvc_vae.h): argument marshalling only; the convolutions and the
blend run in the HIP kernels of libregenvc_attn.so on torch's current stream.

Activations are channels-last bf16 [T, H, W, C] (the plane) or
[n_tiles, T, Hr, Wr, C] (the tiles' buffers); convolution weights bf16
[Cout, 3, 3, 3, Cin], biases bf16 [Cout].
"""
from __future__ import annotations

import ctypes
from typing import List, Sequence, Tuple

import torch

from . import _lib


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def split(H: int, W: int, ty: int, tx: int, halo: int):
    """Tiles of a ty x tx split with the given halo (regenvc_vae_split):
    returns (ctypes array of VaeTile, Hr, Wr); host-only."""
    tiles = (_lib.VaeTile * (ty * tx))()
    hr, wr = ctypes.c_int32(), ctypes.c_int32()
    st = _lib.load().regenvc_vae_split(H, W, ty, tx, halo, tiles, ctypes.byref(hr), ctypes.byref(wr))
    _lib.check(st, "regenvc_vae_split")
    return tiles, hr.value, wr.value


def _check(t: torch.Tensor, name: str):
    if t.device.type != "cuda" or t.dtype != torch.bfloat16 or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous bf16 device tensor")


_N_CU = {}


def conv3d_workspace_bytes(T: int, Hr: int, Wr: int, n_tiles: int, Cin: int, Cout: int, device) -> int:
    """Workspace bytes of the split-K form of one convolution on this device
    (regenvc_vae_conv3d_workspace; host-only, 0 when it does not split)."""
    idx = torch.device(device).index
    idx = torch.cuda.current_device() if idx is None else idx
    if idx not in _N_CU:
        _N_CU[idx] = torch.cuda.get_device_properties(idx).multi_processor_count
    out = ctypes.c_int64()
    st = _lib.load().regenvc_vae_conv3d_workspace(T, Hr, Wr, n_tiles, Cin, Cout, _N_CU[idx], ctypes.byref(out))
    _lib.check(st, "regenvc_vae_conv3d_workspace")
    return out.value


def conv3d(x: torch.Tensor, w: torch.Tensor, b: torch.Tensor, tiles, Hr: int, Wr: int, plane_hw=None,
           silu: bool = False, split_k: bool = True) -> torch.Tensor:
    """One causal 3D convolution over the listed tiles' regions
    (regenvc_vae_conv3d_fwd).  x: the plane [T, H, W, Cin] (plane_hw None),
    or the tiles' buffers [n, T, Hr, Wr, Cin] (plane_hw = (H, W), the plane's
    size).  Returns [n, T, Hr, Wr, Cout].  split_k: hand the library the
    workspace of its split-K form (a torch allocation), used when the tiles
    alone would leave the GPU mostly idle."""
    for name, t in (("x", x), ("w", w), ("b", b)):
        _check(t, name)
    n = len(tiles)
    if plane_hw is None:
        T, H, W, Cin = x.shape
        is_plane = 1
    else:
        if x.shape[0] != n or tuple(x.shape[2:4]) != (Hr, Wr):
            raise ValueError("tile buffers must be [n_tiles, T, Hr, Wr, C]")
        T, Cin = x.shape[1], x.shape[4]
        H, W = plane_hw
        is_plane = 0
    Cout = w.shape[0]
    if tuple(w.shape) != (Cout, 3, 3, 3, Cin) or tuple(b.shape) != (Cout,):
        raise ValueError("w must be [Cout, 3, 3, 3, Cin] and b [Cout]")
    out = torch.empty((n, T, Hr, Wr, Cout), dtype=torch.bfloat16, device=x.device)
    arr = (_lib.VaeTile * n)(*tiles)
    need = conv3d_workspace_bytes(T, Hr, Wr, n, Cin, Cout, x.device) if split_k else 0
    ws = torch.empty(need, dtype=torch.uint8, device=x.device) if need > 0 else None
    st = _lib.load().regenvc_vae_conv3d_fwd(x.data_ptr(), is_plane, w.data_ptr(), b.data_ptr(), int(silu),
                                            out.data_ptr(), T, H, W, Cin, Cout, arr, n, Hr, Wr,
                                            ws.data_ptr() if ws is not None else None, need, _stream(x.device))
    _lib.check(st, "regenvc_vae_conv3d_fwd")
    return out


def blend(tiles_out: torch.Tensor, tiles, H: int, W: int, band: int) -> torch.Tensor:
    """Blended gather of the tiles' outputs [n, T, Hr, Wr, C] into the plane
    [T, H, W, C] (regenvc_vae_blend)."""
    _check(tiles_out, "tiles_out")
    n, T, Hr, Wr, C = tiles_out.shape
    out = torch.empty((T, H, W, C), dtype=torch.bfloat16, device=tiles_out.device)
    arr = (_lib.VaeTile * n)(*tiles)
    st = _lib.load().regenvc_vae_blend(tiles_out.data_ptr(), arr, n, Hr, Wr, T, H, W, C, band, out.data_ptr(),
                                       _stream(tiles_out.device))
    _lib.check(st, "regenvc_vae_blend")
    return out


def tile_stack(x: torch.Tensor, layers: Sequence[Tuple[torch.Tensor, torch.Tensor]], tiles, Hr: int,
               Wr: int) -> torch.Tensor:
    """The convolution stack (SiLU between layers) on the listed tiles'
    regions of the plane x [T, H, W, C]; returns their outputs
    [n, T, Hr, Wr, C]."""
    T, H, W, _ = x.shape
    y = x
    for i, (w, b) in enumerate(layers):
        y = conv3d(y, w, b, tiles, Hr, Wr, plane_hw=None if i == 0 else (H, W), silu=i + 1 < len(layers))
    return y


def split_stack(x: torch.Tensor, layers, ty: int, tx: int, halo: int, band: int) -> torch.Tensor:
    """The whole split VAE stage on one GPU: every tile's stack (one batched
    launch per layer), then the blended gather; returns [T, H, W, C]."""
    T, H, W, _ = x.shape
    tiles, Hr, Wr = split(H, W, ty, tx, halo)
    tl = list(tiles)
    return blend(tile_stack(x, layers, tl, Hr, Wr), tl, H, W, band)
