// Internal launch interface of the spatially split VAE tile kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace regenvc {

constexpr int kVaeMaxTiles = 16;

// One tile of the split plane: its core and its region (core widened by the
// halo, clipped to the plane), half-open row / column ranges.
struct VaeTile {
    int32_t core_y0, core_y1, core_x0, core_x1;
    int32_t reg_y0, reg_y1, reg_x0, reg_x1;
};

// Causal 3D convolution of every listed tile's region, as an implicit GEMM:
// out[t][y][x][o] = act(b[o] + sum_{dt,dy,dx,c} in[t-2+dt][y-1+dy][x-1+dx][c]
// w[o][dt][dy][dx][c]) per tile, zeros before frame 0 and outside the tile's
// region.  Input: the plane [T, H, W, Cin] (regions index into it), or the
// tiles' own buffers [n][T][Hr][Wr][Cin] (a previous layer's output).
// Output: [n][T][Hr][Wr][Cout] (positions past a region's size unused).
struct ConvArgs {
    const void *in;
    const void *w;     // bf16 [Cout, 3, 3, 3, Cin]
    const void *bias;  // bf16 [Cout]
    void *out;
    int32_t T, H, W, Cin, Cout, Hr, Wr, n_tiles;
    int32_t in_is_plane, silu;
    VaeTile tiles[kVaeMaxTiles];
    void *ws;          // split-K partials (f32), or null: no split
    int64_t ws_bytes;
};
// K ranges a launch of M output rows uses with ws_bytes of workspace (1: none).
int conv_splits(int64_t M, int N, int Cin, int n_cu, int64_t ws_bytes);
// Workspace bytes that give a launch its full split (0: it does not split).
size_t conv_workspace_bytes(int64_t M, int N, int Cin, int n_cu);
hipError_t launch_vae_conv(const ConvArgs &a, hipStream_t stream);

// Blended gather of the tiles' outputs [n][T][Hr][Wr][C] into the plane
// [T, H, W, C] (bf16) with separable linear ramps of half-width `band`
// across every seam between cores.
struct BlendArgs {
    const void *tiles_out;
    void *out;
    int32_t T, H, W, C, Hr, Wr, n_tiles, band;
    VaeTile tiles[kVaeMaxTiles];
};
hipError_t launch_vae_blend(const BlendArgs &a, hipStream_t stream);

}  // namespace regenvc
