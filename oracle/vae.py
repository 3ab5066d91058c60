"""Reference oracle of the spatially split VAE tile -- TEST INFRASTRUCTURE ONLY.

Plain float64 numpy (a matmul per kernel tap is the library step); the
product neither imports nor calls this module.

What is computed (paper Sec. 3.6, spatially split VAE decode and encode):
the VAE's latent (or image) plane is cut into tiles, one per GPU; each GPU
runs the VAE's convolutions on its tile widened by a halo sized to the
receptive field, and the gathered tiles are blended where they overlap, so
that no seam shows.  The paper prints neither the layers nor the blend; the
readings taken here:

  layers   causal 3D convolutions over (frame, row, column), as in a video
           VAE: output frame t sees input frames t-2, t-1, t (zeros before
           the first frame) and a 3 x 3 spatial neighbourhood (zeros outside
           the convolved region); bias, and SiLU between layers; activations
           channels-last [T, H, W, C], stored as bf16 after every layer
  tiles    the H x W plane cut into ty x tx rectangular cores (near-equal
           rows and columns); a tile's region is its core widened by `halo`
           on every side that faces another tile (clipped to the plane), and
           the tile runs the whole stack on that region alone (its borders
           padded with zeros, like the plane's)
  blend    separable linear ramps: along each axis, across a band of 2 * b
           pixels centred on every seam between two cores, the weight of
           the tile on one side falls linearly from 1 to 0 while the other's
           rises, w = (b + s) / (2 b) clipped to [0, 1] with s the
           signed distance from the seam to the pixel's centre, positive
           inside the tile's own core; b <= halo and 2 b <= the narrowest
           core (the two seams' bands of a core must not overlap); a pixel's
           output is
           sum_i w_i(row) w_i(col) out_i -- the weights of the tiles covering
           a pixel sum to 1
With halo >= b + (layers) -- the blend band plus the stack's receptive
radius -- every value that receives weight is computed from true input
pixels, and the blended result equals the stack on the whole plane.
"""
from __future__ import annotations

import numpy as np

from .dit import round_bf16, silu, widen


def conv3d_causal(x: np.ndarray, w: np.ndarray, b: np.ndarray) -> np.ndarray:
    """x [T, H, W, Cin]; w [Cout, 3, 3, 3, Cin] (taps dt, dy, dx: input frame
    t - 2 + dt, row y - 1 + dy, column x - 1 + dx); b [Cout].  Zeros before
    the first frame and outside the plane.  Returns [T, H, W, Cout]."""
    T, H, W, _ = x.shape
    xp = np.zeros((T + 2, H + 2, W + 2, x.shape[3]))
    xp[2:, 1:H + 1, 1:W + 1] = x
    Cin, Cout = x.shape[3], w.shape[0]
    out = np.zeros((T * H * W, Cout))
    for dt in range(3):
        for dy in range(3):
            for dx in range(3):
                tap = xp[dt:dt + T, dy:dy + H, dx:dx + W].reshape(T * H * W, Cin)
                out += tap @ w[:, dt, dy, dx, :].T
    return out.reshape(T, H, W, Cout) + b


def stack(x: np.ndarray, layers) -> np.ndarray:
    """The convolution stack: layers = [(w, b), ...] as bf16 bits; SiLU
    between layers (not after the last); every layer's output stored as
    bf16.  x: bf16 values (float64) [T, H, W, C]."""
    for i, (w, b) in enumerate(layers):
        y = conv3d_causal(x, widen(w), widen(b))
        if i + 1 < len(layers):
            y = silu(y)
        x = round_bf16(y)
    return x


def split(n: int, parts: int):
    """Boundaries of `parts` near-equal cores along an axis of n pixels."""
    return [(i * n) // parts for i in range(parts + 1)]


def tile_regions(H: int, W: int, ty: int, tx: int, halo: int):
    """[(core rows, core cols, region rows, region cols)] per tile, each a
    half-open (start, stop) pair; regions widen the cores by `halo` on the
    sides facing another tile."""
    ys, xs = split(H, ty), split(W, tx)
    out = []
    for i in range(ty):
        for j in range(tx):
            r0 = ys[i] - (halo if i > 0 else 0)
            r1 = ys[i + 1] + (halo if i + 1 < ty else 0)
            c0 = xs[j] - (halo if j > 0 else 0)
            c1 = xs[j + 1] + (halo if j + 1 < tx else 0)
            out.append(((ys[i], ys[i + 1]), (xs[j], xs[j + 1]), (max(r0, 0), min(r1, H)), (max(c0, 0), min(c1, W))))
    return out


def ramp(n: int, core, region, band: int) -> np.ndarray:
    """Blend weight of a tile along one axis at pixels region[0] .. region[1]-1
    (see the module docstring); 1 everywhere if band = 0 inside the core."""
    p = np.arange(region[0], region[1]) + 0.5   # pixel centres
    w = np.ones(len(p))
    if band == 0:
        return ((p >= core[0]) & (p < core[1])).astype(np.float64)
    if core[0] > 0:      # seam at core[0]: s = p - core[0]
        w = np.minimum(w, np.clip((band + (p - core[0])) / (2 * band), 0, 1))
    if core[1] < n:      # seam at core[1]: s = core[1] - p
        w = np.minimum(w, np.clip((band + (core[1] - p)) / (2 * band), 0, 1))
    return w


def tiled(x: np.ndarray, layers, ty: int, tx: int, halo: int, band: int):
    """Every tile's stack on its own region, then the blended gather.
    Returns (blended output [T, H, W, Cout], per-tile outputs)."""
    T, H, W, _ = x.shape
    if band > halo:
        raise ValueError("the blend band cannot be wider than the halo")
    if 2 * band > min(H // ty, W // tx):
        raise ValueError("the blend bands of a core's two seams would overlap (2 band > core size)")
    tiles = []
    out = None
    for core_r, core_c, reg_r, reg_c in tile_regions(H, W, ty, tx, halo):
        y = stack(x[:, reg_r[0]:reg_r[1], reg_c[0]:reg_c[1]], layers)
        tiles.append(y)
        if out is None:
            out = np.zeros((T, H, W, y.shape[3]))
        wgt = np.outer(ramp(H, core_r, reg_r, band), ramp(W, core_c, reg_c, band))
        out[:, reg_r[0]:reg_r[1], reg_c[0]:reg_c[1]] += wgt[None, :, :, None] * y
    return out, tiles
