/*
 * regenvc_vae.h -- C ABI of the gfx950 kernels of the spatially split VAE
 * (paper Sec. 3.6): the VAE's latent or image plane is cut into tiles, one
 * per GPU; each GPU runs the VAE's convolutions on its tile widened by a
 * halo sized to the receptive field, and the gathered tiles are blended
 * where they overlap so that no seam shows.
 *
 * The paper prints neither the layers nor the blend; the readings:
 *   - layers: causal 3D convolutions over (frame, row, column), as in a
 *     video VAE: output frame t sees input frames t-2, t-1, t (zeros before
 *     the first frame) and a 3 x 3 neighbourhood (zeros outside the tile's
 *     region); bias, optionally SiLU; channels-last bf16 activations
 *     [T, H, W, C], weights bf16 [Cout, 3, 3, 3, Cin] (taps dt, dy, dx),
 *     accumulation fp32, outputs rounded to bf16;
 *   - tiles: the H x W plane cut into ty x tx near-equal cores; a tile's
 *     region is its core widened by `halo` on every side facing another tile,
 *     clipped to the plane (regenvc_vae_split);
 *   - blend: separable linear ramps -- along each axis, across a band of
 *     2 b pixels centred on each seam between two cores, a tile's weight is
 *     (b + s) / (2 b) clipped to [0, 1], s the signed distance from the seam
 *     to the pixel centre, positive inside the tile's core; weights of the
 *     tiles covering a pixel sum to 1.  With halo >= b + (number of layers),
 *     the blended result equals the layers run on the whole plane.
 *
 * Conventions are those of regenvc_attn.h.  None of these calls allocates.
 */
#ifndef REGENVC_VAE_H
#define REGENVC_VAE_H

#include <stdint.h>

#include "regenvc_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

#define REGENVC_VAE_MAX_TILES 16

/* One tile: core rows [core_y0, core_y1) x columns [core_x0, core_x1), and
   its region (core + halo, clipped to the plane), half-open. */
typedef struct {
    int32_t core_y0, core_y1, core_x0, core_x1;
    int32_t reg_y0, reg_y1, reg_x0, reg_x1;
} regenvc_vae_tile;

/* Splits an H x W plane into ty x tx tiles (row-major: tile i*tx + j is core
   row i, column j) with the given halo; cores are [k n / parts, (k+1) n /
   parts) along each axis.  Writes ty*tx descriptors to `tiles` and the
   largest region height / width to *Hr / *Wr (the per-tile buffer shape).
   ty*tx <= REGENVC_VAE_MAX_TILES; halo >= 0; every core at least 1 x 1.
   Host-only. */
regenvc_status regenvc_vae_split(int32_t H, int32_t W, int32_t ty, int32_t tx, int32_t halo,
                                 regenvc_vae_tile *tiles, int32_t *Hr, int32_t *Wr);

/* One causal 3D convolution layer on the regions of n_tiles tiles (one
   GPU's share is one tile; a single GPU may run all of them in one call).
     in:  in_is_plane != 0: the plane, bf16 [T, H, W, Cin] (contiguous), the
          regions cut from it; in_is_plane == 0: the tiles' own buffers,
          bf16 [n_tiles][T][Hr][Wr][Cin] (a previous layer's output)
     w: bf16 [Cout, 3, 3, 3, Cin]; bias: bf16 [Cout]; silu != 0 applies SiLU
     out: bf16 [n_tiles][T][Hr][Wr][Cout]; a tile's values at rows >=
          region height or columns >= region width are unspecified
     workspace: NULL, or caller-owned DEVICE memory of workspace_bytes
          (256-byte aligned, not overlapping any other argument) for the
          split-K form: when the output tiles would leave most compute units
          idle (one GPU's single tile), K is cut into ranges whose f32
          partial sums go to the workspace and a second kernel adds them,
          the bias and the activation.  Up to
          regenvc_vae_conv3d_workspace bytes are used; less gives fewer
          ranges, NULL (or too little for two) none.  The result is the same
          up to fp32 summation order.  Nothing is allocated.
   Cin, Cout multiples of 64; T >= 1; 1 <= n_tiles <= REGENVC_VAE_MAX_TILES;
   every region inside the plane, no larger than Hr x Wr; pointers 16-byte
   aligned; out must not overlap in, w or bias. */
regenvc_status regenvc_vae_conv3d_fwd(const void *in, int32_t in_is_plane, const void *w, const void *bias,
                                      int32_t silu, void *out, int32_t T, int32_t H, int32_t W, int32_t Cin,
                                      int32_t Cout, const regenvc_vae_tile *tiles, int32_t n_tiles,
                                      int32_t Hr, int32_t Wr, void *workspace, int64_t workspace_bytes,
                                      void *stream);

/* Workspace bytes that let regenvc_vae_conv3d_fwd of this shape use its
   full split-K form on a device with n_cu compute units (0: it does not
   split).  Host-only; T, Hr, Wr, n_tiles >= 1, Cin and Cout multiples of
   64, n_cu >= 1. */
regenvc_status regenvc_vae_conv3d_workspace(int32_t T, int32_t Hr, int32_t Wr, int32_t n_tiles, int32_t Cin,
                                            int32_t Cout, int32_t n_cu, int64_t *bytes);

/* Blended gather: out (bf16 [T, H, W, C]) = sum over the tiles covering each
   pixel of ramp_row x ramp_col x tile value, from the tiles' outputs bf16
   [n_tiles][T][Hr][Wr][C].  The tiles must be those of one regenvc_vae_split
   (their cores tiling the plane); 0 <= band <= halo and 2 band <= the
   smallest core side (band 0 is a plain crop to the cores).  C a multiple of
   8; pointers 16-byte aligned; out must not overlap tiles_out. */
regenvc_status regenvc_vae_blend(const void *tiles_out, const regenvc_vae_tile *tiles, int32_t n_tiles,
                                 int32_t Hr, int32_t Wr, int32_t T, int32_t H, int32_t W, int32_t C,
                                 int32_t band, void *out, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* REGENVC_VAE_H */
