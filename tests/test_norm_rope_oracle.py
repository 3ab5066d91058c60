"""Pins of the oracle's q/k RMSNorm + 3D rotary embedding (CPU only).

The oracle (oracle_norm_rope) is the definition written out; these tests pin
it to properties that do not restate its formula: the norm's closed forms and
invariances, the rotation's norm preservation, the dependence of q.k on
relative positions only, the axis layout at unit frequency (theta = 1), and
the frequency schedule at a theta for which it is a power of two.  A copy of
the oracle with a planted mistake must fail at least one of them.
"""
import math
import os
import shutil
import tempfile

import numpy as np
import pytest

import oracle
from oracle import build as oracle_build
from paper_2607_28144_amd import synth

F32 = lambda v: float(np.float32(v))  # noqa: E731
D, H = 128, 2
PF, PH, PW = 22, 21, 21   # pairs per axis at D = 128 (frame, row, column)
GRID = (3, 4, 5)          # frames x rows x cols


def rnd(seed, shape, scale=1.0):
    return synth.normal_bf16(np.random.default_rng(seed), shape, scale)


def ones_w(n):
    return synth.f32_to_bf16_bits(np.ones(n, dtype=np.float32))


def axis_of_pair(i):
    return 0 if i < PF else (1 if i < PF + PH else 2)


def pos_of(g, grid=GRID):
    return (g // (grid[1] * grid[2]), (g // grid[2]) % grid[1], g % grid[2])


def test_position_zero_is_rmsnorm_closed_form(lib=None):
    """Token 0 sits at (0, 0, 0): no rotation.  With w = 1 and eps = 0 the
    output is x scaled to unit mean square over all H*D channels."""
    x = rnd(1, (1, 1, H, D), 3.0)
    y = oracle.norm_rope(x, ones_w(H * D), GRID, eps=0.0, lib=lib)
    xf = synth.bf16_bits_to_f32(x).astype(np.float64)
    assert abs(np.mean(y ** 2) - 1.0) < 1e-12
    ratio = y / xf
    np.testing.assert_allclose(ratio, ratio.flat[0], rtol=1e-12)


def test_large_eps_closed_form(lib=None):
    """eps dominating the mean square: r -> 1/sqrt(eps + ms), checked at eps = 1e6."""
    x = rnd(2, (1, 1, H, D))
    w = rnd(3, (H * D,))
    y = oracle.norm_rope(x, w, GRID, eps=1e6, lib=lib)
    xf = synth.bf16_bits_to_f32(x).astype(np.float64)
    wf = synth.bf16_bits_to_f32(w).astype(np.float64)
    ms = np.mean(xf ** 2)
    np.testing.assert_allclose(y[0, 0], (xf[0, 0] * wf.reshape(H, D)) / math.sqrt(ms + 1e6), rtol=1e-12)


def test_scale_invariance_and_weight_linearity(lib=None):
    x = rnd(4, (2, 7, H, D))
    w = rnd(5, (H * D,))
    x4 = synth.f32_to_bf16_bits(synth.bf16_bits_to_f32(x) * 4)   # exact in bf16
    w2 = synth.f32_to_bf16_bits(synth.bf16_bits_to_f32(w) * 2)
    y = oracle.norm_rope(x, w, GRID, eps=0.0, lib=lib)
    np.testing.assert_allclose(oracle.norm_rope(x4, w, GRID, eps=0.0, lib=lib), y, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(oracle.norm_rope(x, w2, GRID, eps=0.0, lib=lib), 2 * y, rtol=1e-12, atol=1e-14)


def test_rotation_preserves_pair_norms(lib=None):
    """The same token values placed at every position of the grid: each
    (2i, 2i+1) pair keeps its length (position 0 gives the unrotated one)."""
    n = GRID[0] * GRID[1] * GRID[2]
    one = rnd(6, (1, 1, H, D))
    x = np.ascontiguousarray(np.broadcast_to(one, (1, n, H, D)))
    y = oracle.norm_rope(x, rnd(7, (H * D,)), GRID, lib=lib)
    norms = y[..., 0::2] ** 2 + y[..., 1::2] ** 2
    np.testing.assert_allclose(norms, np.broadcast_to(norms[:, :1], norms.shape), rtol=1e-12, atol=1e-14)
    assert not np.allclose(y[0, 1], y[0, 0])  # ... and it does rotate


def test_scores_depend_on_relative_positions_only(lib=None):
    """q at position p and k at p': per head q.k is unchanged when both move by
    the same amount along any one axis."""
    grid = (5, 6, 7)
    wq, wk = rnd(8, (H * D,)), rnd(9, (H * D,))
    qv, kv = rnd(10, (1, 1, H, D)), rnd(11, (1, 1, H, D))

    def score(gq, gk):
        yq = oracle.norm_rope(qv, wq, grid, token0=gq, lib=lib)[0, 0]
        yk = oracle.norm_rope(kv, wk, grid, token0=gk, lib=lib)[0, 0]
        return np.sum(yq * yk, axis=-1)

    def g(f, r, c):
        return (f * grid[1] + r) * grid[2] + c

    base = score(g(1, 2, 3), g(0, 1, 1))
    for shift in ((2, 0, 0), (0, 3, 0), (0, 0, 3), (1, 1, 2)):
        moved = score(g(1 + shift[0], 2 + shift[1], 3 + shift[2]), g(shift[0], 1 + shift[1], 1 + shift[2]))
        np.testing.assert_allclose(moved, base, rtol=1e-10, atol=1e-12)
    assert not np.allclose(score(g(1, 2, 3), g(0, 0, 0)), base)  # the relative position matters


def test_axis_layout_at_unit_frequency(lib=None):
    """theta = 1: every pair turns by its axis position (radians).  A token
    whose pairs are all (s, 0) must come out as (s cos p, s sin p) with p the
    frame, row or column of the token for the first 22, next 21 and last 21
    pairs respectively."""
    xf = np.zeros((1, 1, H, D), dtype=np.float32)
    xf[..., 0::2] = 1.0
    x = synth.f32_to_bf16_bits(xf)
    s = math.sqrt(2.0)  # mean square of x is 1/2
    for g in (0, 1, 7, 23, 41, 59):
        y = oracle.norm_rope(x, ones_w(H * D), GRID, token0=g, eps=0.0, theta=1.0, lib=lib)[0, 0]
        pos = pos_of(g)
        for i in range(D // 2):
            p = pos[axis_of_pair(i)]
            np.testing.assert_allclose(y[:, 2 * i], s * math.cos(p), atol=1e-12)
            np.testing.assert_allclose(y[:, 2 * i + 1], s * math.sin(p), atol=1e-12)


def test_frequency_schedule_at_power_of_two_theta(lib=None):
    """theta = 2^(d_a/2) makes pair k of an axis with d_a dims turn at
    frequency 2^-k: one step along that axis turns it by exactly 2^-k."""
    xf = np.zeros((1, 1, H, D), dtype=np.float32)
    xf[..., 0::2] = 1.0
    x = synth.f32_to_bf16_bits(xf)
    s = math.sqrt(2.0)
    first = {0: 0, 1: PF, 2: PF + PH}
    npairs = {0: PF, 1: PH, 2: PW}
    step = {0: GRID[1] * GRID[2], 1: GRID[2], 2: 1}  # token index one step along each axis
    for axis in (0, 1, 2):
        theta = 2.0 ** npairs[axis]   # = 2^(d_a / 2)
        y = oracle.norm_rope(x, ones_w(H * D), GRID, token0=step[axis], eps=0.0, theta=theta, lib=lib)[0, 0]
        for kk in range(npairs[axis]):
            i = first[axis] + kk
            ang = 2.0 ** -kk
            np.testing.assert_allclose(y[:, 2 * i], s * math.cos(ang), atol=1e-12)
            np.testing.assert_allclose(y[:, 2 * i + 1], s * math.sin(ang), atol=1e-12)


PINS = [test_position_zero_is_rmsnorm_closed_form, test_large_eps_closed_form,
        test_scale_invariance_and_weight_linearity, test_rotation_preserves_pair_norms,
        test_scores_depend_on_relative_positions_only, test_axis_layout_at_unit_frequency,
        test_frequency_schedule_at_power_of_two_theta]


def _pins_hold(lib) -> bool:
    for pin in PINS:
        try:
            pin(lib=lib)
        except AssertionError:
            return False
    return True


MUTANTS = [
    ("eps dropped", "const double r = 1.0 / sqrt(ss / C + eps);", "const double r = 1.0 / sqrt(ss / C);"),
    ("mean over one head", "const double r = 1.0 / sqrt(ss / C + eps);", "const double r = 1.0 / sqrt(ss / D + eps);"),
    ("weight of the wrong head", "bf16_to_double(w[h * D + d]);", "bf16_to_double(w[d]);"),
    ("sine sign flipped", "yr[2 * i] = a0 * c - a1 * sn;", "yr[2 * i] = a0 * c + a1 * sn;"),
    ("pair members swapped", "yr[2 * i + 1] = a0 * sn + a1 * c;", "yr[2 * i + 1] = a1 * sn + a0 * c;"),
    ("frequency exponent halved", "pow(theta, -2.0 * kk / (2.0 * pairs))", "pow(theta, -1.0 * kk / (2.0 * pairs))"),
    ("axes row/column swapped", "(double)((g / grid_w) % grid_h),\n                                   (double)(g % grid_w)};",
     "(double)(g % grid_w),\n                                   (double)((g / grid_w) % grid_h)};"),
    ("row from the wrong divisor", "(double)((g / grid_w) % grid_h)", "(double)((g / grid_h) % grid_w)"),
    ("frame pairs one short", "if (i < pf) {", "if (i < pf - 1) {"),
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistakes_are_caught(name, old, new):
    src = open(os.path.join(oracle.ORACLE_DIR, "oracle.c")).read()
    assert src.count(old) == 1, f"mutation site for '{name}' not found exactly once"
    tmp = tempfile.mkdtemp(prefix="norm_rope_mutant_")
    try:
        # a file name no other loaded library has: the dynamic loader may hand
        # back an already loaded object for a path or file it has seen before
        tag = "".join(ch if ch.isalnum() else "_" for ch in name)
        path = os.path.join(tmp, f"norm_rope_mutant_{tag}.c")
        with open(path, "w") as f:
            f.write(src.replace(old, new))
        lib = oracle.open_library(oracle_build.build(source=path, out=path[:-2] + ".so"))
        assert not _pins_hold(lib), f"planted mistake '{name}' was not caught by the pins"
    finally:
        shutil.rmtree(tmp, ignore_errors=True)


def test_real_oracle_holds_every_pin():
    assert _pins_hold(oracle._load())
