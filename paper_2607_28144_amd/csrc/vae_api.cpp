// C ABI of the spatially split VAE tile kernels (include/regenvc_vae.h):
// host-side tile split, synchronous validation, launches on the caller's
// stream.  Nothing here allocates.
#include "regenvc_vae.h"

#include <hip/hip_runtime.h>

#include <algorithm>

#include "abi_util.hpp"
#include "vae_kernels.hpp"

using regenvc::abi::aligned;
using regenvc::abi::failf;
using regenvc::abi::overlaps;
using regenvc::abi::range_of;

static_assert(REGENVC_VAE_MAX_TILES == regenvc::kVaeMaxTiles, "header and library agree");
static_assert(sizeof(regenvc_vae_tile) == sizeof(regenvc::VaeTile), "same tile record");

namespace {

// The tiles must describe a split of the plane: cores inside it, regions
// containing their cores, inside the plane and no larger than Hr x Wr.
regenvc_status check_tiles(const char *fn, const regenvc_vae_tile *t, int32_t n, int32_t H, int32_t W, int32_t Hr,
                           int32_t Wr)
{
    if (t == nullptr) return failf(REGENVC_ERR_INVALID_ARG, "%s: tiles is NULL", fn);
    if (n < 1 || n > REGENVC_VAE_MAX_TILES)
        return failf(REGENVC_ERR_INVALID_ARG, "%s: n_tiles=%d not in [1, %d]", fn, n, REGENVC_VAE_MAX_TILES);
    for (int i = 0; i < n; ++i) {
        const regenvc_vae_tile &a = t[i];
        const bool ok = 0 <= a.reg_y0 && a.reg_y0 <= a.core_y0 && a.core_y0 < a.core_y1 && a.core_y1 <= a.reg_y1 &&
                        a.reg_y1 <= H && 0 <= a.reg_x0 && a.reg_x0 <= a.core_x0 && a.core_x0 < a.core_x1 &&
                        a.core_x1 <= a.reg_x1 && a.reg_x1 <= W && a.reg_y1 - a.reg_y0 <= Hr &&
                        a.reg_x1 - a.reg_x0 <= Wr;
        if (!ok) return failf(REGENVC_ERR_INVALID_ARG, "%s: tile %d is not a core inside a region of the plane", fn, i);
    }
    return REGENVC_OK;
}

void copy_tiles(regenvc::VaeTile *dst, const regenvc_vae_tile *src, int n)
{
    for (int i = 0; i < n; ++i)
        dst[i] = regenvc::VaeTile{src[i].core_y0, src[i].core_y1, src[i].core_x0, src[i].core_x1,
                                  src[i].reg_y0,  src[i].reg_y1,  src[i].reg_x0,  src[i].reg_x1};
}

}  // namespace

extern "C" {

regenvc_status regenvc_vae_split(int32_t H, int32_t W, int32_t ty, int32_t tx, int32_t halo, regenvc_vae_tile *tiles,
                                 int32_t *Hr, int32_t *Wr)
{
    const char *fn = "regenvc_vae_split";
    if (!tiles || !Hr || !Wr) return failf(REGENVC_ERR_INVALID_ARG, "%s: a NULL output", fn);
    if (ty < 1 || tx < 1 || ty * tx > REGENVC_VAE_MAX_TILES || halo < 0 || H < ty || W < tx)
        return failf(REGENVC_ERR_INVALID_ARG, "%s: bad split %d x %d of %d x %d (halo %d)", fn, ty, tx, H, W, halo);
    int hr = 0, wr = 0;
    for (int i = 0; i < ty; ++i)
        for (int j = 0; j < tx; ++j) {
            regenvc_vae_tile &t = tiles[i * tx + j];
            t.core_y0 = (int32_t)((int64_t)i * H / ty);
            t.core_y1 = (int32_t)((int64_t)(i + 1) * H / ty);
            t.core_x0 = (int32_t)((int64_t)j * W / tx);
            t.core_x1 = (int32_t)((int64_t)(j + 1) * W / tx);
            t.reg_y0 = std::max(0, t.core_y0 - (i > 0 ? halo : 0));
            t.reg_y1 = std::min(H, t.core_y1 + (i + 1 < ty ? halo : 0));
            t.reg_x0 = std::max(0, t.core_x0 - (j > 0 ? halo : 0));
            t.reg_x1 = std::min(W, t.core_x1 + (j + 1 < tx ? halo : 0));
            hr = std::max(hr, t.reg_y1 - t.reg_y0);
            wr = std::max(wr, t.reg_x1 - t.reg_x0);
        }
    *Hr = hr;
    *Wr = wr;
    regenvc::abi::clear_error();
    return REGENVC_OK;
}

regenvc_status regenvc_vae_conv3d_fwd(const void *in, int32_t in_is_plane, const void *w, const void *bias,
                                      int32_t silu, void *out, int32_t T, int32_t H, int32_t W, int32_t Cin,
                                      int32_t Cout, const regenvc_vae_tile *tiles, int32_t n_tiles, int32_t Hr,
                                      int32_t Wr, void *workspace, int64_t workspace_bytes, void *stream)
{
    const char *fn = "regenvc_vae_conv3d_fwd";
    if (T < 1 || H < 1 || W < 1 || Hr < 1 || Wr < 1)
        return failf(REGENVC_ERR_INVALID_ARG, "%s: bad sizes (T=%d H=%d W=%d Hr=%d Wr=%d)", fn, T, H, W, Hr, Wr);
    if (Cin < 64 || Cout < 64 || Cin % 64 || Cout % 64)
        return failf(REGENVC_ERR_UNSUPPORTED, "%s: channels Cin=%d Cout=%d must be multiples of 64", fn, Cin, Cout);
    regenvc_status st = check_tiles(fn, tiles, n_tiles, H, W, Hr, Wr);
    if (st != REGENVC_OK) return st;
    if (!in || !w || !bias || !out) return failf(REGENVC_ERR_INVALID_ARG, "%s: a NULL pointer", fn);
    if (!aligned(in, 16) || !aligned(w, 16) || !aligned(bias, 16) || !aligned(out, 16))
        return failf(REGENVC_ERR_UNSUPPORTED, "%s: pointers must be 16-byte aligned", fn);
    const int64_t tile_pix = (int64_t)T * Hr * Wr;
    if ((int64_t)n_tiles * tile_pix > 0x7fffffff)
        return failf(REGENVC_ERR_UNSUPPORTED, "%s: more than 2^31 - 1 output pixels", fn);
    const int64_t in_bytes = (in_is_plane ? (int64_t)T * H * W : n_tiles * tile_pix) * Cin * 2;
    const auto ro = range_of(out, n_tiles * tile_pix * Cout * 2);
    if (overlaps(ro, range_of(in, in_bytes)) || overlaps(ro, range_of(w, (int64_t)Cout * 27 * Cin * 2)) ||
        overlaps(ro, range_of(bias, (int64_t)Cout * 2)))
        return failf(REGENVC_ERR_INVALID_ARG, "%s: out overlaps an input", fn);
    if (workspace != nullptr) {
        if (workspace_bytes < 0) return failf(REGENVC_ERR_INVALID_ARG, "%s: workspace_bytes < 0", fn);
        if (!aligned(workspace, 256))
            return failf(REGENVC_ERR_UNSUPPORTED, "%s: workspace must be 256-byte aligned", fn);
        const auto rw = range_of(workspace, workspace_bytes);
        if (overlaps(rw, ro) || overlaps(rw, range_of(in, in_bytes)) ||
            overlaps(rw, range_of(w, (int64_t)Cout * 27 * Cin * 2)) || overlaps(rw, range_of(bias, (int64_t)Cout * 2)))
            return failf(REGENVC_ERR_INVALID_ARG, "%s: workspace overlaps another argument", fn);
    }
    if ((st = regenvc::abi::device_ok()) != REGENVC_OK) return st;
    regenvc::ConvArgs a{};
    a.in = in, a.w = w, a.bias = bias, a.out = out;
    a.T = T, a.H = H, a.W = W, a.Cin = Cin, a.Cout = Cout, a.Hr = Hr, a.Wr = Wr, a.n_tiles = n_tiles;
    a.in_is_plane = in_is_plane != 0, a.silu = silu != 0;
    a.ws = workspace, a.ws_bytes = workspace != nullptr ? workspace_bytes : 0;
    copy_tiles(a.tiles, tiles, n_tiles);
    return regenvc::abi::launch_status(regenvc::launch_vae_conv(a, static_cast<hipStream_t>(stream)), fn);
}

regenvc_status regenvc_vae_conv3d_workspace(int32_t T, int32_t Hr, int32_t Wr, int32_t n_tiles, int32_t Cin,
                                            int32_t Cout, int32_t n_cu, int64_t *bytes)
{
    const char *fn = "regenvc_vae_conv3d_workspace";
    if (bytes == nullptr) return failf(REGENVC_ERR_INVALID_ARG, "%s: bytes is NULL", fn);
    if (T < 1 || Hr < 1 || Wr < 1 || n_tiles < 1 || n_tiles > REGENVC_VAE_MAX_TILES || n_cu < 1)
        return failf(REGENVC_ERR_INVALID_ARG, "%s: bad sizes (T=%d Hr=%d Wr=%d n_tiles=%d n_cu=%d)", fn, T, Hr, Wr,
                     n_tiles, n_cu);
    if (Cin < 64 || Cout < 64 || Cin % 64 || Cout % 64)
        return failf(REGENVC_ERR_UNSUPPORTED, "%s: channels Cin=%d Cout=%d must be multiples of 64", fn, Cin, Cout);
    *bytes = (int64_t)regenvc::conv_workspace_bytes((int64_t)n_tiles * T * Hr * Wr, Cout, Cin, n_cu);
    regenvc::abi::clear_error();
    return REGENVC_OK;
}

regenvc_status regenvc_vae_blend(const void *tiles_out, const regenvc_vae_tile *tiles, int32_t n_tiles, int32_t Hr,
                                 int32_t Wr, int32_t T, int32_t H, int32_t W, int32_t C, int32_t band, void *out,
                                 void *stream)
{
    const char *fn = "regenvc_vae_blend";
    if (T < 1 || H < 1 || W < 1 || Hr < 1 || Wr < 1 || C < 8 || C % 8)
        return failf(REGENVC_ERR_INVALID_ARG, "%s: bad sizes (T=%d H=%d W=%d C=%d)", fn, T, H, W, C);
    regenvc_status st = check_tiles(fn, tiles, n_tiles, H, W, Hr, Wr);
    if (st != REGENVC_OK) return st;
    int min_core = 1 << 30;
    for (int i = 0; i < n_tiles; ++i)
        min_core = std::min({min_core, tiles[i].core_y1 - tiles[i].core_y0, tiles[i].core_x1 - tiles[i].core_x0});
    if (band < 0 || 2 * band > min_core)
        return failf(REGENVC_ERR_INVALID_ARG, "%s: band=%d (0 <= band, 2 band <= smallest core side %d)", fn, band,
                     min_core);
    for (int i = 0; i < n_tiles; ++i) {
        // every side facing another tile needs at least `band` of halo
        const regenvc_vae_tile &t = tiles[i];
        if ((t.core_y0 > 0 && t.core_y0 - t.reg_y0 < band) || (t.core_y1 < H && t.reg_y1 - t.core_y1 < band) ||
            (t.core_x0 > 0 && t.core_x0 - t.reg_x0 < band) || (t.core_x1 < W && t.reg_x1 - t.core_x1 < band))
            return failf(REGENVC_ERR_INVALID_ARG, "%s: tile %d has less halo than the band %d", fn, i, band);
    }
    if (!tiles_out || !out) return failf(REGENVC_ERR_INVALID_ARG, "%s: a NULL pointer", fn);
    if (!aligned(tiles_out, 16) || !aligned(out, 16))
        return failf(REGENVC_ERR_UNSUPPORTED, "%s: pointers must be 16-byte aligned", fn);
    if (overlaps(range_of(out, (int64_t)T * H * W * C * 2), range_of(tiles_out, (int64_t)n_tiles * T * Hr * Wr * C * 2)))
        return failf(REGENVC_ERR_INVALID_ARG, "%s: out overlaps tiles_out", fn);
    if ((st = regenvc::abi::device_ok()) != REGENVC_OK) return st;
    regenvc::BlendArgs a{};
    a.tiles_out = tiles_out, a.out = out;
    a.T = T, a.H = H, a.W = W, a.C = C, a.Hr = Hr, a.Wr = Wr, a.n_tiles = n_tiles, a.band = band;
    copy_tiles(a.tiles, tiles, n_tiles);
    return regenvc::abi::launch_status(regenvc::launch_vae_blend(a, static_cast<hipStream_t>(stream)), fn);
}

}  // extern "C"
