"""Pins of the split-VAE tile oracle (oracle/vae.py) on the CPU:

  conv3d_causal  pure-Python brute force of the definition on a tiny case;
                 the centre tap of the current frame as an identity kernel;
                 a kernel with only the oldest-frame tap shifts frames by 2;
                 causality (changing frame t0 moves no earlier output);
                 the count of in-plane taps at corners, edges and interior
                 (an all-ones kernel on all-ones input)
  stack          two identity layers give SiLU once (between the layers)
  blend          weights non-negative and summing to 1 over the tiles that
                 cover each pixel, for several splits, halos and bands;
                 across a seam the two tiles' ramps mirror each other;
                 cores tile each axis, sizes differing by at most one
  tiled          with halo >= band + layers the blended tiles equal the
                 stack on the whole plane; with band 0 (plain crop) and
                 halo >= layers likewise; with a halo of only the band, the
                 seams differ (the halo must cover the receptive field)
and planted mistakes, each of which must fail one of these pins.
"""
import itertools
import types

import numpy as np
import pytest

from oracle import vae
from oracle.dit import widen
from paper_2607_28144_amd import synth


def rnd(seed, shape, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def pin_brute_force(m):
    T, H, W, Ci, Co = 3, 4, 5, 2, 3
    x, w, b = rnd(1, (T, H, W, Ci)), rnd(2, (Co, 3, 3, 3, Ci)), rnd(3, (Co,))
    want = np.zeros((T, H, W, Co))
    for t, y, xx, o in itertools.product(range(T), range(H), range(W), range(Co)):
        acc = b[o]
        for dt, dy, dx, c in itertools.product(range(3), range(3), range(3), range(Ci)):
            tt, yy, xs = t - 2 + dt, y - 1 + dy, xx - 1 + dx
            if tt >= 0 and 0 <= yy < H and 0 <= xs < W:
                acc += x[tt, yy, xs, c] * w[o, dt, dy, dx, c]
        want[t, y, xx, o] = acc
    return bool(np.allclose(m.conv3d_causal(x, w, b), want, rtol=0, atol=1e-12))


def pin_identity_and_shift(m):
    x = rnd(4, (4, 5, 6, 3))
    w = np.zeros((3, 3, 3, 3, 3))
    for c in range(3):
        w[c, 2, 1, 1, c] = 1.0            # current frame, centre pixel
    ok = np.array_equal(m.conv3d_causal(x, w, np.zeros(3)), x)
    w2 = np.zeros((3, 3, 3, 3, 3))
    for c in range(3):
        w2[c, 0, 1, 1, c] = 1.0           # two frames back
    y = m.conv3d_causal(x, w2, np.zeros(3))
    ok &= np.array_equal(y[2:], x[:-2]) and not np.any(y[:2])
    return bool(ok)


def pin_causality(m):
    x = rnd(5, (5, 4, 4, 2))
    w, b = rnd(6, (2, 3, 3, 3, 2)), rnd(7, (2,))
    y = m.conv3d_causal(x, w, b)
    x2 = x.copy()
    x2[3] += 10.0
    y2 = m.conv3d_causal(x2, w, b)
    return bool(np.array_equal(y[:3], y2[:3]) and not np.allclose(y[3], y2[3]))


def pin_tap_counts(m):
    T, H, W = 3, 4, 5
    y = m.conv3d_causal(np.ones((T, H, W, 1)), np.ones((1, 3, 3, 3, 1)), np.zeros(1))[..., 0]
    frames = np.array([1, 2, 3])                         # frames available to t = 0, 1, 2
    rows = np.array([2, 3, 3, 2])                        # rows available to y = 0 .. 3
    cols = np.array([2, 3, 3, 3, 2])
    return bool(np.array_equal(y, frames[:, None, None] * rows[None, :, None] * cols[None, None, :]))


def pin_partition_of_unity(m):
    ok = True
    for H, W, ty, tx, halo, band in [(60, 104, 2, 4, 4, 2), (60, 104, 2, 4, 2, 2), (17, 23, 3, 2, 5, 3),
                                     (12, 16, 2, 2, 3, 0), (9, 9, 3, 3, 1, 1)]:
        total = np.zeros((H, W))
        for core_r, core_c, reg_r, reg_c in m.tile_regions(H, W, ty, tx, halo):
            wr, wc = m.ramp(H, core_r, reg_r, band), m.ramp(W, core_c, reg_c, band)
            ok &= bool(np.all(wr >= 0) and np.all(wc >= 0))
            total[reg_r[0]:reg_r[1], reg_c[0]:reg_c[1]] += np.outer(wr, wc)
        ok &= bool(np.allclose(total, 1.0, rtol=0, atol=1e-12))
    return ok


def pin_stack_activation(m):
    """Two identity layers (centre tap of the current frame, zero bias): the
    stack is SiLU once, between the layers, rounded to bf16."""
    x = synth.bf16_bits_to_f32(synth.normal_bf16(np.random.default_rng(9), (2, 3, 4, 2))).astype(np.float64)
    w = np.zeros((2, 3, 3, 3, 2), dtype=np.float32)
    for c in range(2):
        w[c, 2, 1, 1, c] = 1.0
    layer = (synth.f32_to_bf16_bits(w), synth.f32_to_bf16_bits(np.zeros(2, dtype=np.float32)))
    want = m.round_bf16(x / (1.0 + np.exp(-x)))
    return bool(np.array_equal(m.stack(x, [layer, layer]), want))


def pin_split_and_ramp_shape(m):
    """Cores tile each axis with sizes differing by at most one, and across a
    seam the two tiles' ramps are mirror images of each other."""
    ok = True
    for n, parts in [(60, 2), (104, 4), (17, 3), (9, 2)]:
        b = m.split(n, parts)
        sizes = np.diff(b)
        ok &= b[0] == 0 and b[-1] == n and sizes.max() - sizes.min() <= 1
    n, band = 10, 2
    wi = m.ramp(n, (0, 5), (0, 7), band)          # tile below the seam at 5
    wj = m.ramp(n, (5, 10), (3, 10), band)        # tile above it
    ok &= bool(np.allclose(wi[3:7], wj[:4][::-1]) and np.allclose(wi[3:7] + wj[:4], 1.0))
    return bool(ok)


def small_stack(seed=8):
    x, convs = synth.vae_inputs(seed, 3, 12, 16, 8)
    return widen(x), convs


def pin_tiled_equals_whole(m):
    x, convs = small_stack()
    full = m.stack(x, convs)
    ok = True
    for ty, tx, halo, band in [(2, 2, 4, 2), (2, 3, 2, 0), (3, 2, 5, 2)]:
        out, _ = m.tiled(x, convs, ty, tx, halo, band)
        ok &= bool(np.allclose(out, full, rtol=0, atol=1e-12))
    out, _ = m.tiled(x, convs, 2, 2, 2, 2)      # halo = band: no room for the receptive field
    ok &= bool(np.abs(out - full).max() > 1e-3)
    try:
        m.tiled(x, convs, 3, 2, 5, 3)            # bands of one core's two seams would overlap
        ok = False
    except ValueError:
        pass
    return ok


PINS = [pin_brute_force, pin_identity_and_shift, pin_causality, pin_tap_counts, pin_partition_of_unity,
        pin_stack_activation, pin_split_and_ramp_shape, pin_tiled_equals_whole]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_pins(pin):
    assert pin(vae)


MUTANTS = [
    ("future frames instead of past", "xp[2:, 1:H + 1, 1:W + 1] = x", "xp[:T, 1:H + 1, 1:W + 1] = x"),
    ("kernel not transposed", "out += tap @ w[:, dt, dy, dx, :].T", "out += tap @ w[:, dt, dy, dx, :]"),
    ("bias dropped", "return out.reshape(T, H, W, Cout) + b", "return out.reshape(T, H, W, Cout)"),
    ("activation after the last layer too", "if i + 1 < len(layers):", "if True:"),
    ("no activation", "y = silu(y)", "y = y"),
    ("ramp half as wide", "np.clip((band + (p - core[0])) / (2 * band), 0, 1)",
     "np.clip((band + (p - core[0])) / band, 0, 1)"),
    ("ramp from the pixel edge, not its centre", "p = np.arange(region[0], region[1]) + 0.5",
     "p = np.arange(region[0], region[1]) + 0.0"),
    ("halo only below", "r0 = ys[i] - (halo if i > 0 else 0)", "r0 = ys[i]"),
    ("uneven cores", "return [(i * n) // parts for i in range(parts + 1)]",
     "return [min(n, i * (n // parts + 1)) for i in range(parts + 1)]"),
]


def load_mutant(old, new):
    src = open(vae.__file__).read()
    assert src.count(old) == 1, old
    mod = types.ModuleType("oracle._vae_mutant")
    mod.__package__ = "oracle"
    mod.__file__ = vae.__file__
    exec(compile(src.replace(old, new), vae.__file__ + " (mutant)", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistakes_are_caught(name, old, new):
    m = load_mutant(old, new)

    def holds(pin):
        try:
            with np.errstate(all="ignore"):
                return pin(m)
        except Exception:
            return False
    assert not all(holds(p) for p in PINS), f"mutant '{name}' passes every pin"
