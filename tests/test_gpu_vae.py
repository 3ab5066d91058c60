"""GPU parity of the spatially split VAE tile (include/regenvc_vae.h) against
the fp64 oracle (oracle/vae.py) on the same seeded bf16 inputs.

Each stage is checked on the GPU's own bf16 input to it, so that every bound
is the per-element one of a single rounding: a convolution output satisfies
|gpu - ref| <= 2^-8 |ref| + 2 * 2^-20 * sum |x||w| (fp32 accumulation over
the 27 Cin taps; SiLU's slope is below 1.1), the blend 2^-8 |ref| + 1e-6.
The end-to-end result (all stages on the GPU) is compared with the oracle's
stack on the whole plane -- equal in exact arithmetic when the halo covers
band + layers -- within two bf16 steps of each value plus 2^-8 of the RMS,
room for the rare rounding flips that carry from one layer into the next.
"""
import ctypes

import numpy as np
import pytest

from oracle import vae as ovae
from oracle.dit import widen
from paper_2607_28144_amd import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

ULP = 2.0 ** -8
ACC = 2.0 ** -20


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_28144_amd import vae  # noqa: F401  (fails loudly if the library is missing)
    yield
    torch.cuda.synchronize()


def kern():
    from paper_2607_28144_amd import vae
    return vae


def dev_bits(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def host(t):
    return t.float().cpu().numpy().astype(np.float64)


def check_bound(name, got, ref, tol):
    err = np.abs(got - ref)
    over = int(np.count_nonzero(err > tol))
    print(f"[vae] {name}: max|d|={err.max():.3e} rms={np.sqrt((err * err).mean()):.3e} "
          f"max err/bound={float((err / tol).max()):.3f} over={over}/{err.size}", flush=True)
    assert np.all(np.isfinite(got)) and over == 0, name


def region(t):
    return (t.reg_y0, t.reg_y1), (t.reg_x0, t.reg_x1)


def conv_ref(x, w_bits, b_bits, silu):
    """Oracle convolution of bf16-valued x (one region) and its bound."""
    W, B = widen(w_bits), widen(b_bits)
    y = ovae.conv3d_causal(x, W, B)
    slack = 2 * ACC * ovae.conv3d_causal(np.abs(x), np.abs(W), np.zeros_like(B))
    if silu:
        y = ovae.silu(y)
        slack = 1.1 * slack
    return y, ULP * np.abs(y) + slack + 1e-6


def stagewise(name, T, H, W, C, ty, tx, halo, band, tiles_to_check, seed):
    x, convs = synth.vae_inputs(seed, T, H, W, C)
    X = widen(x)
    tiles, Hr, Wr = kern().split(H, W, ty, tx, halo)
    tl = list(tiles)
    dx = dev_bits(x)
    dconvs = [(dev_bits(w), dev_bits(b)) for w, b in convs]
    y1 = kern().conv3d(dx, *dconvs[0], tl, Hr, Wr, silu=True)
    y2 = kern().conv3d(y1, *dconvs[1], tl, Hr, Wr, plane_hw=(H, W))
    out = kern().blend(y2, tl, H, W, band)
    torch.cuda.synchronize()
    g1, g2 = host(y1), host(y2)
    for i in tiles_to_check:
        (r0, r1), (c0, c1) = region(tl[i])
        h, w = r1 - r0, c1 - c0
        ref, tol = conv_ref(X[:, r0:r1, c0:c1], *convs[0], True)
        check_bound(f"{name} tile {i} conv 1 (SiLU)", g1[i, :, :h, :w], ref, tol)
        ref, tol = conv_ref(g1[i, :, :h, :w], *convs[1], False)
        check_bound(f"{name} tile {i} conv 2", g2[i, :, :h, :w], ref, tol)
    ref = np.zeros((T, H, W, C))
    for i, t in enumerate(tl):
        (r0, r1), (c0, c1) = region(t)
        wgt = np.outer(ovae.ramp(H, (t.core_y0, t.core_y1), (r0, r1), band),
                       ovae.ramp(W, (t.core_x0, t.core_x1), (c0, c1), band))
        ref[:, r0:r1, c0:c1] += wgt[None, :, :, None] * g2[i, :, :r1 - r0, :c1 - c0]
    check_bound(f"{name} blend", host(out), ref, ULP * np.abs(ref) + 1e-6)
    return X, convs, dx, dconvs, tl, Hr, Wr, y1, y2, out


def test_small_plane_every_tile_and_the_whole_plane():
    """3 frames of 12 x 16, 64 channels, 2 x 2 tiles, halo 4 >= band 2 + 2
    layers: every tile's stages, the blend, and the blended result against
    the oracle's stack on the whole plane."""
    X, convs, *_, out = stagewise("small", 3, 12, 16, 64, 2, 2, 4, 2, range(4), 71)
    full = ovae.stack(X, convs)
    got = host(out)
    check_bound("small end to end vs whole plane", got, full,
                2 * ULP * np.abs(full) + ULP * float(np.sqrt((full * full).mean())))


def test_window_latent_tile_of_an_eight_way_split():
    """The decoder stage at the window's latent resolution: 7 frames of
    60 x 104, 384 channels, split 2 x 4 (one tile per GPU of the node), halo
    4, band 2.  Tiles 1 (top row, inner column) and 4 (bottom-left) are
    checked stage by stage; one tile launched alone (one GPU's share) gives
    bitwise the batched launch's values when K is not split, and passes the
    same per-element bounds in its split-K form (the single tile's 64 row
    tiles run as 4 K ranges each); the blend is checked everywhere."""
    T, H, W, C = 7, 60, 104, 384
    X, convs, dx, dconvs, tl, Hr, Wr, y1, y2, out = stagewise("window", T, H, W, C, 2, 4, 4, 2, (1, 4), 72)
    assert kern().conv3d_workspace_bytes(T, Hr, Wr, 1, C, C, dx.device) > 0  # the single tile splits K
    assert kern().conv3d_workspace_bytes(T, Hr, Wr, 8, C, C, dx.device) == 0  # the batch does not
    one1 = kern().conv3d(dx, *dconvs[0], [tl[1]], Hr, Wr, silu=True, split_k=False)
    one2 = kern().conv3d(one1, *dconvs[1], [tl[1]], Hr, Wr, plane_hw=(H, W), split_k=False)
    sk1 = kern().conv3d(dx, *dconvs[0], [tl[1]], Hr, Wr, silu=True)
    sk2 = kern().conv3d(sk1, *dconvs[1], [tl[1]], Hr, Wr, plane_hw=(H, W))
    torch.cuda.synchronize()
    (r0, r1), (c0, c1) = region(tl[1])
    h, w = r1 - r0, c1 - c0
    assert torch.equal(one1[0, :, :h, :w], y1[1, :, :h, :w])
    assert torch.equal(one2[0, :, :h, :w], y2[1, :, :h, :w])
    g1 = host(sk1)[0, :, :h, :w]
    ref, tol = conv_ref(X[:, r0:r1, c0:c1], *convs[0], True)
    check_bound("window tile 1 split-K conv 1 (SiLU)", g1, ref, tol)
    ref, tol = conv_ref(g1, *convs[1], False)
    check_bound("window tile 1 split-K conv 2", host(sk2)[0, :, :h, :w], ref, tol)


def test_split_k_every_range_count():
    """Small convolutions in the split-K form with workspaces that allow 2,
    3 and 8 K ranges (and none): each against the oracle's per-element
    bound, on a 1 x 2 split (two tiles, 64 channels in, 128 out)."""
    T, H, W, Cin, Cout = 3, 9, 14, 64, 128
    rng = np.random.default_rng(74)
    x = synth.normal_bf16(rng, (T, H, W, Cin))
    wb = synth.normal_bf16(rng, (Cout, 3, 3, 3, Cin), float(1.0 / np.sqrt(27 * Cin)))
    bb = synth.normal_bf16(rng, (Cout,), 0.02)
    X = widen(x)
    tiles, Hr, Wr = kern().split(H, W, 1, 2, 3)
    tl = list(tiles)
    M = len(tl) * T * Hr * Wr
    dx, dw, db = dev_bits(x), dev_bits(wb), dev_bits(bb)
    from paper_2607_28144_amd import _lib
    lib = _lib.load()
    arr = (_lib.VaeTile * len(tl))(*tl)
    for ranges in (0, 2, 3, 8):
        out = torch.empty((len(tl), T, Hr, Wr, Cout), dtype=torch.bfloat16, device=dx.device)
        nbytes = ranges * M * Cout * 4
        ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dx.device) if ranges else None
        st = lib.regenvc_vae_conv3d_fwd(dx.data_ptr(), 1, dw.data_ptr(), db.data_ptr(), 1, out.data_ptr(), T, H, W,
                                        Cin, Cout, arr, len(tl), Hr, Wr, ws.data_ptr() if ws is not None else None,
                                        nbytes, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        _lib.check(st, "regenvc_vae_conv3d_fwd")
        torch.cuda.synchronize()
        g = host(out)
        for i in range(len(tl)):
            (r0, r1), (c0, c1) = region(tl[i])
            ref, tol = conv_ref(X[:, r0:r1, c0:c1], wb, bb, True)
            check_bound(f"split-K {ranges} ranges, tile {i}", g[i, :, :r1 - r0, :c1 - c0], ref, tol)


def test_plain_crop_and_single_tile():
    """band 0 (plain crop to the cores) and a 1 x 1 split (no halo at all: the
    stack on the whole plane) against the oracle."""
    T, H, W, C = 2, 10, 12, 64
    x, convs = synth.vae_inputs(73, T, H, W, C)
    X = widen(x)
    dconvs = [(dev_bits(w), dev_bits(b)) for w, b in convs]
    for ty, tx, halo, band in [(1, 1, 0, 0), (2, 3, 2, 0)]:
        got = host(kern().split_stack(dev_bits(x), dconvs, ty, tx, halo, band))
        torch.cuda.synchronize()
        full = ovae.stack(X, convs)
        check_bound(f"split {ty}x{tx} halo {halo} band {band} vs whole plane", got, full,
                    2 * ULP * np.abs(full) + ULP * float(np.sqrt((full * full).mean())))
