"""Pins of the block oracle (oracle/dit.py) on the CPU, against what the
mathematics fixes rather than the oracle's own formulas:

  gemm          exact integer products (pure-Python sums and int64 matmul)
  gelu_tanh     gelu(0) = 0; gelu(x) - gelu(-x) = x (the odd part of the
                tanh form is x/2); limits x and 0 at large |x|; within the
                approximation error (4.7e-4 at most) of the exact x * Phi(x)
                (math.erf)
  silu          silu(x) - silu(-x) = x; silu(0) = 0
  layer_norm    zero mean and unit variance (eps = 0), invariance under
                x -> a x + b (a > 0), the affine map applied after
  rms_norm      unit root mean square (eps = 0, w = 1), scale invariance
  round_bf16    equals the bit-level float32 -> bf16 rounder of the input
                generator on float32 values, ties included
  modulation    W = 0 gives the bias; shift = scale = 0 is the identity
  block         zero gates and a zero cross-attention projection give the
                identity; with two tokens and two context tokens every
                softmax has the two-key closed form (sigmoid of the score
                difference), so the block is recomputed here as a chain of
                linear maps, norms, GELU and that closed form, without the
                oracle's attention; joint permutation of the context tokens
                leaves the output unchanged
and a set of planted mistakes (each a one-line change of a copy of the
oracle module) that must each fail one of these pins.
"""
import math
import types

import numpy as np
import pytest

import oracle
from oracle import dit
from paper_2607_28144_amd import synth

C = dit.C




@pytest.fixture(scope="module")
def params():
    return synth.dit_params(11)


# ------------------------------------------------------------------ elementwise pieces
def pin_gemm_integers(m):
    rng = np.random.default_rng(1)
    a = rng.integers(-8, 9, size=(5, 7))
    w = rng.integers(-8, 9, size=(3, 7))
    b = rng.integers(-8, 9, size=(3,))
    ref = [[sum(int(a[i, k]) * int(w[j, k]) for k in range(7)) + int(b[j]) for j in range(3)] for i in range(5)]
    ok = np.array_equal(m.gemm(a.astype(np.float64), w.astype(np.float64), b.astype(np.float64)), np.array(ref))
    a2 = rng.integers(-16, 17, size=(64, 300))
    w2 = rng.integers(-16, 17, size=(40, 300))
    ok &= np.array_equal(m.gemm(a2.astype(np.float64), w2.astype(np.float64)), a2.astype(np.int64) @ w2.T)
    return ok


def pin_gelu(m):
    x = np.linspace(-12, 12, 2001)
    ok = m.gelu_tanh(np.array([0.0]))[0] == 0.0
    ok &= np.allclose(m.gelu_tanh(x) - m.gelu_tanh(-x), x, rtol=0, atol=1e-14)
    ok &= abs(m.gelu_tanh(np.array([40.0]))[0] - 40.0) < 1e-12 and abs(m.gelu_tanh(np.array([-40.0]))[0]) < 1e-12
    exact = np.array([xi * 0.5 * (1 + math.erf(xi / math.sqrt(2))) for xi in x])
    ok &= np.abs(m.gelu_tanh(x) - exact).max() < 5e-4
    return bool(ok)


def pin_silu(m):
    x = np.linspace(-30, 30, 601)
    return bool(m.silu(np.array([0.0]))[0] == 0.0 and np.allclose(m.silu(x) - m.silu(-x), x, rtol=0, atol=1e-12))


def pin_layer_norm(m):
    rng = np.random.default_rng(2)
    x = rng.standard_normal((6, C)) * 3 + 1.5
    y = m.layer_norm(x, 0.0)
    ok = np.allclose(y.mean(axis=1), 0, atol=1e-12) and np.allclose((y * y).mean(axis=1), 1, atol=1e-12)
    ok &= np.allclose(m.layer_norm(2.5 * x - 7.0, 0.0), y, atol=1e-12)
    w, b = rng.standard_normal(C), rng.standard_normal(C)
    ok &= np.allclose(m.layer_norm(x, 0.0, w, b), y * w + b, atol=1e-12)
    # eps enters the variance: a constant row offset by d normalizes to d / sqrt(d^2 + eps)
    row = np.zeros((1, C))
    row[0, :C // 2], row[0, C // 2:] = 1e-3, -1e-3
    ok &= np.allclose(m.layer_norm(row, 1e-6), row / math.sqrt(1e-6 + 1e-6), atol=1e-12)
    return bool(ok)


def pin_rms_norm(m):
    rng = np.random.default_rng(3)
    x = rng.standard_normal((6, C)) * 2.0
    y = m.rms_norm(x, np.ones(C), 0.0)
    ok = np.allclose(np.sqrt((y * y).mean(axis=1)), 1, atol=1e-12) and np.allclose(m.rms_norm(4 * x, np.ones(C), 0.0), y)
    row = np.full((1, C), 1e-3)
    ok &= np.allclose(m.rms_norm(row, np.ones(C), 1e-6), row / math.sqrt(1e-6 + 1e-6), atol=1e-12)
    return bool(ok)


def pin_round_bf16(m):
    rng = np.random.default_rng(4)
    f = (rng.standard_normal(20000) * np.exp(rng.uniform(-20, 20, 20000))).astype(np.float32)
    # exact ties: float32 values halfway between two bf16 values
    ties = ((rng.integers(0x3f80, 0x4100, 500).astype(np.uint32) << 16) | 0x8000).view(np.float32)
    f = np.concatenate([f, ties, -ties, np.float32([0.0, 1.0, -2.5])])
    want = synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(f)).astype(np.float64)
    return bool(np.array_equal(m.round_bf16(f.astype(np.float64)), want))


def pin_modulation(m):
    rng = np.random.default_rng(5)
    e = rng.standard_normal(C)
    b = rng.standard_normal(6 * C)
    ok = np.array_equal(m.modulation(e, np.zeros((6 * C, C)), b), b.reshape(6, C))
    w = rng.standard_normal((6 * C, C))
    e0 = np.zeros(C)  # silu(0) = 0: the weights do not enter
    ok &= np.array_equal(m.modulation(e0, w, b), b.reshape(6, C))
    y = rng.standard_normal((3, C))
    ok &= np.array_equal(m.modulate(y, np.zeros(C), np.zeros(C)), y)
    ok &= np.allclose(m.modulate(y, np.full(C, 2.0), np.full(C, 0.5)), 1.5 * y + 2.0)
    return bool(ok)


# ------------------------------------------------------------------ block
def pin_block_identity(m, params):
    """Gates g1 = g2 = 0 (their rows of W_mod and b_mod) and a zero
    cross-attention output projection: every branch adds exactly zero."""
    p = dict(params)
    w_mod = synth.bf16_bits_to_f32(p["w_mod"]).reshape(6, C, C).copy()
    b_mod = synth.bf16_bits_to_f32(p["b_mod"]).reshape(6, C).copy()
    w_mod[[2, 5]] = 0
    b_mod[[2, 5]] = 0
    p["w_mod"] = synth.f32_to_bf16_bits(w_mod.reshape(6 * C, C))
    p["b_mod"] = synth.f32_to_bf16_bits(b_mod.reshape(6 * C))
    p["w_oc"] = np.zeros_like(p["w_oc"])
    p["b_oc"] = np.zeros_like(p["b_oc"])
    x, e, kc, vc = synth.dit_inputs(6, 8, 5, steps=1)
    y = m.block(x.astype(np.float64), e[0], p, kc, vc, (2, 2, 2))
    return bool(np.array_equal(y, x.astype(np.float64)))


def chain_two_tokens(x, e, p, kc, vc, grid):
    """The block for TWO tokens and TWO context tokens, with every attention
    written as the two-key closed form: per head, the weights of keys 0 and
    1 are sigmoid(s0 - s1) and sigmoid(s1 - s0) of the scaled scores.  q/k
    normalization and rotation use oracle.norm_rope (pinned on its own);
    nothing else of the block oracle is used."""
    W = {n: dit.widen(v) for n, v in p.items()}
    r = dit.round_bf16
    scale = float(np.float32(1.0 / math.sqrt(dit.HEAD_DIM)))
    H, D = dit.HEADS, dit.HEAD_DIM
    mod = (W["w_mod"] @ (e / (1.0 + np.exp(-e))) + W["b_mod"]).reshape(6, C)

    def ln(z, w=None, b=None):
        mu = z.mean(axis=1, keepdims=True)
        z = (z - mu) / np.sqrt(((z - mu) ** 2).mean(axis=1, keepdims=True) + 1e-6)
        return z * (1 if w is None else w) + (0 if b is None else b)

    def two_key_attention(q, k, v):  # q [2, C]; k, v [2, H, D] -> [2, C]
        out = np.zeros((2, H, D))
        for i in range(2):
            for h in range(H):
                s0 = scale * q[i, h * D:(h + 1) * D] @ k[0, h]
                s1 = scale * q[i, h * D:(h + 1) * D] @ k[1, h]
                a0 = 1.0 / (1.0 + math.exp(s1 - s0))
                out[i, h] = a0 * v[0, h] + (1.0 - a0) * v[1, h]
        return r(out.reshape(2, C))

    def bits(z):
        return dit.to_bits(z).reshape(1, 2, H, D)

    x = x.astype(np.float64)
    h1 = r(ln(x) * (1 + mod[1]) + mod[0])
    q = r(h1 @ W["w_qkv"][:C].T + W["b_qkv"][:C])
    k = r(h1 @ W["w_qkv"][C:2 * C].T + W["b_qkv"][C:2 * C])
    v = r(h1 @ W["w_qkv"][2 * C:].T + W["b_qkv"][2 * C:])
    q = r(oracle.norm_rope(bits(q), p["w_qn"], grid, 0, 1e-6, 10000.0)).reshape(2, C)
    k = r(oracle.norm_rope(bits(k), p["w_kn"], grid, 0, 1e-6, 10000.0)).reshape(2, H, D)
    a = two_key_attention(q, k, v.reshape(2, H, D))
    x = x + mod[2] * (a @ W["w_o"].T + W["b_o"])
    h2 = r(ln(x, W["w_n3"], W["b_n3"]))
    qc = r(h2 @ W["w_qc"].T + W["b_qc"])
    qc = r(qc / np.sqrt((qc * qc).mean(axis=1, keepdims=True) + 1e-6) * W["w_qcn"])
    c = two_key_attention(qc, dit.widen(kc), dit.widen(vc))
    x = x + (c @ W["w_oc"].T + W["b_oc"])
    h3 = r(ln(x) * (1 + mod[4]) + mod[3])
    u = h3 @ W["w_1"].T + W["b_1"]
    f = r(0.5 * u * (1 + np.tanh(math.sqrt(2 / math.pi) * (u + 0.044715 * u ** 3))))
    return x + mod[5] * (f @ W["w_2"].T + W["b_2"])


def pin_block_two_tokens(m, params):
    """Tokens at columns 0 and 1 of a 1 x 1 x 2 grid, two context tokens."""
    x, e, kc, vc = synth.dit_inputs(7, 2, 2, steps=1)
    y = m.block(x.astype(np.float64), e[0], params, kc, vc, (1, 1, 2))
    want = chain_two_tokens(x, e[0].astype(np.float64), params, kc, vc, (1, 1, 2))
    return bool(np.allclose(y, want, rtol=0, atol=1e-9))


def pin_block_context_permutation(m, params):
    x, e, kc, vc = synth.dit_inputs(8, 8, 9, steps=1)
    y = m.block(x.astype(np.float64), e[0], params, kc, vc, (2, 2, 2))
    perm = np.random.default_rng(9).permutation(9)
    y2 = m.block(x.astype(np.float64), e[0], params, kc[perm], vc[perm], (2, 2, 2))
    return bool(np.allclose(y, y2, rtol=0, atol=1e-9))


ELEMENTWISE_PINS = [pin_gemm_integers, pin_gelu, pin_silu, pin_layer_norm, pin_rms_norm, pin_round_bf16,
                    pin_modulation]
BLOCK_PINS = [pin_block_identity, pin_block_two_tokens, pin_block_context_permutation]


@pytest.mark.parametrize("pin", ELEMENTWISE_PINS, ids=lambda f: f.__name__)
def test_elementwise_pins(pin):
    assert pin(dit)


@pytest.mark.parametrize("pin", BLOCK_PINS, ids=lambda f: f.__name__)
def test_block_pins(pin, params):
    assert pin(dit, params)


def test_block_keeps_a_random_window_finite_and_moving(params):
    """A sanity check of scale on a 7 x 6 x 8 window over 4 steps (not a pin):
    the residual stream stays finite and every step changes it."""
    x, e, kc, vc = synth.dit_inputs(10, 7 * 6 * 8, 64)
    y = x.astype(np.float64)
    for s in range(4):
        y2 = dit.block(y, e[s], params, kc, vc, (7, 6, 8))
        assert np.all(np.isfinite(y2)) and np.abs(y2 - y).max() > 1e-2
        y = y2


# ------------------------------------------------------------------ planted mistakes
MUTANTS = [
    ("gelu cubic term dropped", "(x + 0.044715 * x ** 3)", "(x)"),
    ("gelu constant sqrt(pi/2)", "np.sqrt(2.0 / np.pi)", "np.sqrt(np.pi / 2.0)"),
    ("silu sign", "x / (1.0 + np.exp(-x))", "x / (1.0 + np.exp(x))"),
    ("layer norm eps dropped", "np.sqrt(var + eps)", "np.sqrt(var)"),
    ("layer norm unbiased variance", "((x - mu) ** 2).mean(axis=-1, keepdims=True)",
     "((x - mu) ** 2).sum(axis=-1, keepdims=True) / (x.shape[-1] - 1)"),
    ("rms norm without the mean", "(x * x).mean(axis=-1, keepdims=True)", "(x * x).sum(axis=-1, keepdims=True)"),
    ("modulate by scale, not 1 + scale", "y * (1.0 + scale) + shift", "y * scale + shift"),
    ("weight not transposed", "np.asarray(w, dtype=np.float64).T)", "np.asarray(w, dtype=np.float64))"),
    ("rounding to 7 significand bits", "np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)",
     "np.ldexp(np.rint(np.ldexp(m, 7)), e - 7)"),
    ("key and value swapped", "q, k, v = qkv[:, :C], qkv[:, C:2 * C], qkv[:, 2 * C:]",
     "q, v, k = qkv[:, :C], qkv[:, C:2 * C], qkv[:, 2 * C:]"),
    ("shift and scale rows swapped", "sh1, sc1, g1, sh2, sc2, g2 = modulation", "sc1, sh1, g1, sh2, sc2, g2 = modulation"),
    ("gate on the cross-attention branch", "x = x + gemm(c, W[\"w_oc\"], W[\"b_oc\"])",
     "x = x + g1 * gemm(c, W[\"w_oc\"], W[\"b_oc\"])"),
    ("feed-forward residual dropped", "return x + g2 * gemm(f, W[\"w_2\"], W[\"b_2\"])",
     "return g2 * gemm(f, W[\"w_2\"], W[\"b_2\"])"),
    ("cross-attention norm without affine", "layer_norm(x, EPS, W[\"w_n3\"], W[\"b_n3\"])", "layer_norm(x, EPS)"),
    ("feed-forward bias dropped", "gelu_tanh(gemm(h3, W[\"w_1\"], W[\"b_1\"]))", "gelu_tanh(gemm(h3, W[\"w_1\"]))"),
]


def load_mutant(old: str, new: str):
    src = open(dit.__file__).read()
    assert src.count(old) == 1, old
    mod = types.ModuleType("oracle._dit_mutant")
    mod.__package__ = "oracle"
    mod.__file__ = dit.__file__
    exec(compile(src.replace(old, new), dit.__file__ + " (mutant)", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistakes_are_caught(name, old, new, params):
    m = load_mutant(old, new)

    def holds(pin, *args):
        try:
            with np.errstate(all="ignore"):
                return pin(m, *args)
        except Exception:  # a shape error is a caught mistake too
            return False
    results = [holds(p) for p in ELEMENTWISE_PINS] + [holds(p, params) for p in BLOCK_PINS]
    assert not all(results), f"mutant '{name}' passes every pin"


def test_row_subset_equals_the_rows_of_the_full_block(params):
    """The rows option restricts the output, not the keys: block(rows=r) is
    block()[r] (a check of the option, not a pin of the definition)."""
    x, e, kc, vc = synth.dit_inputs(13, 2 * 3 * 4, 7, steps=1)
    full = dit.block(x.astype(np.float64), e[0], params, kc, vc, (2, 3, 4))
    rows = [0, 5, 17, 23]
    sub = dit.block(x.astype(np.float64), e[0], params, kc, vc, (2, 3, 4), rows=rows)
    assert np.array_equal(sub, full[rows])
