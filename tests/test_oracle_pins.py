"""Pins of the fp64 oracle to facts fixed by the paper and by mathematics.

The oracle (oracle/oracle.c) is the definition of exact softmax attention
and of the log-sum-exp merge of key/value-chunk partials (paper Sec. 3.5:
under Ulysses each GPU attends over all tokens for its subset of heads;
Ring folds passed-around key/value blocks together with running-max
rescaling; the sharded result is single-device attention apart from the
order of floating-point reductions).  The
paper prints no worked numeric example of attention, so every pin here is
exact mathematics: brute force on tiny inputs, closed forms, invariants, and
a library special case.  test_planted_mistakes_are_caught checks that these
pins would catch plausible mistakes in the oracle.
"""
import math
import os
import shutil
import tempfile

import numpy as np
import pytest

import oracle
import oracle.brute as brute
from oracle import build as oracle_build
from paper_2607_28144_amd import synth

F32 = lambda x: float(np.float32(x))  # noqa: E731  the float32 scale both sides receive


def widen(bits):
    return synth.bf16_bits_to_f32(bits).astype(np.float64)


def ints_bf16(rng, shape, lo, hi):
    """bf16 bits of small integers (exact in bf16, and sums of a few stay exact)."""
    return synth.f32_to_bf16_bits(rng.integers(lo, hi + 1, size=shape).astype(np.float32))


# ---------------------------------------------------------------- brute force
@pytest.mark.parametrize("B,H,Sq,Skv,D,seed", [
    (1, 1, 1, 1, 1, 0), (1, 2, 5, 7, 8, 1), (2, 2, 9, 16, 8, 2), (1, 1, 3, 33, 16, 3), (2, 3, 4, 5, 4, 4)])
def test_oracle_matches_brute_force(B, H, Sq, Skv, D, seed):
    q, k, v = synth.qkv(seed, B, H, Sq, Skv, D)
    scale = F32(1.0 / math.sqrt(D))
    o, lse = oracle.attn(q, k, v, scale)
    O, L = brute.attn(q.tolist(), k.tolist(), v.tolist(), scale)
    np.testing.assert_allclose(o, np.array(O), rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, np.array(L), rtol=0, atol=1e-12)


def test_oracle_matches_brute_force_tiny_config_rows():
    """Tiny config (B=1, H=2, S=256, d=64, seed 1): sampled rows by brute force."""
    q, k, v = synth.qkv(1, 1, 2, 256, 256, 64)
    scale = F32(1.0 / 8.0)
    o, lse = oracle.attn(q, k, v, scale)
    kk, vv = widen(k), widen(v)
    for h in range(2):
        keys = kk[0, :, h, :].tolist()
        vals = vv[0, :, h, :].tolist()
        for i in (0, 1, 127, 200, 255):
            orow, l = brute.attn_row(widen(q[0, i, h, :]).tolist(), keys, vals, scale)
            np.testing.assert_allclose(o[0, i, h], orow, rtol=0, atol=1e-12)
            assert abs(lse[0, h, i] - l) < 1e-12


def test_oracle_matches_torch_sdpa_float64():
    """Library special case: torch's scaled_dot_product_attention in float64 on CPU."""
    torch = pytest.importorskip("torch")
    q, k, v = synth.qkv(1, 1, 2, 256, 256, 64)
    scale = F32(1.0 / 8.0)
    o, _ = oracle.attn(q, k, v, scale)
    tq, tk, tv = (torch.from_numpy(widen(x)).permute(0, 2, 1, 3) for x in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, scale=scale).permute(0, 2, 1, 3).numpy()
    np.testing.assert_allclose(o, ref, rtol=0, atol=1e-12)


# ---------------------------------------------------------------- closed forms
def test_single_key_returns_its_value_row():
    q, k, v = synth.qkv(5, 2, 3, 7, 1, 16)
    scale = F32(0.3)
    o, lse = oracle.attn(q, k, v, scale)
    vv = widen(v)
    for b in range(2):
        for h in range(3):
            for i in range(7):
                assert np.array_equal(o[b, i, h], vv[b, 0, h])  # exactly v_0
                s = scale * math.fsum(widen(q[b, i, h]) * widen(k[b, 0, h]))
                assert abs(lse[b, h, i] - s) < 1e-12


def test_two_keys_sigmoid_closed_form():
    q, k, v = synth.qkv(6, 1, 2, 9, 2, 8)
    scale = F32(0.5)
    o, lse = oracle.attn(q, k, v, scale)
    qq, kk, vv = widen(q), widen(k), widen(v)
    for h in range(2):
        for i in range(9):
            s0 = scale * math.fsum(qq[0, i, h] * kk[0, 0, h])
            s1 = scale * math.fsum(qq[0, i, h] * kk[0, 1, h])
            w0 = 1.0 / (1.0 + math.exp(s1 - s0))
            w1 = 1.0 / (1.0 + math.exp(s0 - s1))
            np.testing.assert_allclose(o[0, i, h], w0 * vv[0, 0, h] + w1 * vv[0, 1, h], rtol=0, atol=1e-13)
            assert abs(lse[0, h, i] - np.logaddexp(s0, s1)) < 1e-12


def test_constant_values_return_that_row():
    rng = np.random.default_rng(7)
    q, k, _ = synth.qkv(7, 1, 2, 11, 40, 16)
    row = synth.normal_bf16(rng, (1, 1, 2, 16))
    v = np.ascontiguousarray(np.broadcast_to(row, (1, 40, 2, 16)))
    o, _ = oracle.attn(q, k, v, F32(0.25))
    np.testing.assert_allclose(o, np.broadcast_to(widen(row), o.shape), rtol=1e-14, atol=0)


@pytest.mark.parametrize("how", ["zero_scale", "zero_q"])
def test_uniform_weights_give_mean_and_log_count(how):
    q, k, v = synth.qkv(8, 1, 2, 5, 37, 8)
    scale = F32(0.2)
    if how == "zero_scale":
        scale = 0.0
    else:
        q = np.zeros_like(q)
    o, lse = oracle.attn(q, k, v, scale)
    vv = widen(v)
    for h in range(2):
        mean = np.array([math.fsum(vv[0, :, h, t]) / 37 for t in range(8)])
        for i in range(5):
            np.testing.assert_allclose(o[0, i, h], mean, rtol=0, atol=1e-15)
            assert abs(lse[0, h, i] - math.log(37)) < 1e-14


# ---------------------------------------------------------------- invariants
def test_joint_key_value_permutation_invariance():
    q, k, v = synth.qkv(9, 1, 2, 13, 50, 16)
    perm = np.random.default_rng(9).permutation(50)
    o1, l1 = oracle.attn(q, k, v, F32(0.25))
    o2, l2 = oracle.attn(q, np.ascontiguousarray(k[:, perm]), np.ascontiguousarray(v[:, perm]), F32(0.25))
    np.testing.assert_allclose(o1, o2, rtol=0, atol=1e-14)
    np.testing.assert_allclose(l1, l2, rtol=0, atol=1e-13)


def test_duplicating_every_key_adds_log2_to_lse():
    q, k, v = synth.qkv(10, 1, 2, 6, 21, 8)
    o1, l1 = oracle.attn(q, k, v, F32(0.3))
    o2, l2 = oracle.attn(q, np.concatenate([k, k], axis=1), np.concatenate([v, v], axis=1), F32(0.3))
    np.testing.assert_allclose(o1, o2, rtol=0, atol=1e-14)
    np.testing.assert_allclose(l2, l1 + math.log(2.0), rtol=0, atol=1e-13)


def test_shifting_every_key_by_u_shifts_lse_by_scaled_q_dot_u():
    rng = np.random.default_rng(11)
    q = ints_bf16(rng, (1, 7, 2, 8), -3, 3)
    k = ints_bf16(rng, (1, 19, 2, 8), -3, 3)
    v = ints_bf16(rng, (1, 19, 2, 8), -4, 4)
    u = rng.integers(-2, 3, size=(1, 1, 2, 8)).astype(np.float32)
    k2 = synth.f32_to_bf16_bits(synth.bf16_bits_to_f32(k) + u)
    scale = 0.125
    o1, l1 = oracle.attn(q, k, v, scale)
    o2, l2 = oracle.attn(q, k2, v, scale)
    np.testing.assert_allclose(o1, o2, rtol=0, atol=1e-13)
    for h in range(2):
        for i in range(7):
            shift = scale * float(np.dot(widen(q[0, i, h]), u[0, 0, h].astype(np.float64)))
            assert abs(l2[0, h, i] - (l1[0, h, i] + shift)) < 1e-12


def test_linearity_in_values_and_convex_hull():
    rng = np.random.default_rng(12)
    q, k, _ = synth.qkv(12, 1, 2, 9, 30, 8)
    v1 = ints_bf16(rng, (1, 30, 2, 8), -8, 8)
    v2 = ints_bf16(rng, (1, 30, 2, 8), -8, 8)
    v3 = synth.f32_to_bf16_bits(2 * synth.bf16_bits_to_f32(v1) - synth.bf16_bits_to_f32(v2))  # exact
    o1, _ = oracle.attn(q, k, v1, F32(0.3))
    o2, _ = oracle.attn(q, k, v2, F32(0.3))
    o3, _ = oracle.attn(q, k, v3, F32(0.3))
    np.testing.assert_allclose(o3, 2 * o1 - o2, rtol=0, atol=1e-12)
    vv = widen(v1)
    lo = vv.min(axis=1, keepdims=True)
    hi = vv.max(axis=1, keepdims=True)
    assert np.all(o1 >= lo - 1e-12) and np.all(o1 <= hi + 1e-12)


def test_lse_between_max_score_and_max_plus_log_count():
    q, k, v = synth.qkv(13, 2, 2, 8, 64, 16)
    scale = F32(0.25)
    _, lse = oracle.attn(q, k, v, scale)
    s = scale * np.einsum("bihd,bjhd->bhij", widen(q), widen(k))
    smax = s.max(axis=-1)
    assert np.all(lse >= smax - 1e-12)
    assert np.all(lse <= smax + math.log(64) + 1e-12)


def test_head_and_batch_subsets_equal_slices_of_the_full_run():
    q, k, v = synth.qkv(14, 3, 4, 10, 17, 8)
    o, lse = oracle.attn(q, k, v, F32(0.35))
    o_sub, l_sub = oracle.attn(q[1:3, :, 1:3], k[1:3, :, 1:3], v[1:3, :, 1:3], F32(0.35))
    assert np.array_equal(o_sub, o[1:3, :, 1:3])
    assert np.array_equal(l_sub, lse[1:3, 1:3])


def test_head_major_strides_equal_token_major():
    q, k, v = synth.qkv(15, 2, 3, 9, 12, 8)
    o, lse = oracle.attn(q, k, v, F32(0.35))
    qt, kt, vt = (np.ascontiguousarray(x.transpose(0, 2, 1, 3)).transpose(0, 2, 1, 3) for x in (q, k, v))
    assert qt.strides != q.strides
    o2, l2 = oracle.attn(qt, kt, vt, F32(0.35))
    assert np.array_equal(o, o2) and np.array_equal(lse, l2)


# ---------------------------------------------------------------- merge
def _chunked(q, k, v, scale, bounds, order=None):
    parts = [oracle.attn(q, np.ascontiguousarray(k[:, a:b]), np.ascontiguousarray(v[:, a:b]), scale)
             for a, b in zip(bounds[:-1], bounds[1:])]
    if order is not None:
        parts = [parts[i] for i in order]
    return oracle.merge([p[0] for p in parts], [p[1] for p in parts])


@pytest.mark.parametrize("bounds", [
    [0, 64, 128, 192, 256],          # even chunks (the ring share splits keys evenly)
    [0, 1, 100, 101, 256],           # uneven, with single-token chunks
    [0, 256],                        # one chunk
    list(range(0, 257, 16)),         # sixteen chunks
])
def test_chunked_partials_merged_equal_unchunked(bounds):
    q, k, v = synth.qkv(16, 1, 2, 20, 256, 16)
    scale = F32(0.25)
    o, lse = oracle.attn(q, k, v, scale)
    om, lm = _chunked(q, k, v, scale, bounds)
    np.testing.assert_allclose(om, o, rtol=0, atol=1e-13)
    np.testing.assert_allclose(lm, lse, rtol=0, atol=1e-12)


def test_merge_is_order_independent():
    q, k, v = synth.qkv(17, 1, 2, 9, 90, 8)
    scale = F32(0.4)
    b = [0, 17, 40, 41, 90]
    o1, l1 = _chunked(q, k, v, scale, b)
    o2, l2 = _chunked(q, k, v, scale, b, order=[3, 1, 0, 2])
    np.testing.assert_allclose(o1, o2, rtol=0, atol=1e-14)
    np.testing.assert_allclose(l1, l2, rtol=0, atol=1e-13)


def test_merge_empty_parts_have_weight_zero_and_all_empty_gives_zero_and_neg_inf():
    q, k, v = synth.qkv(18, 1, 2, 5, 30, 8)
    o, lse = oracle.attn(q, k, v, F32(0.3))
    empty_o = np.zeros_like(o)
    empty_l = np.full_like(lse, -np.inf)
    om, lm = oracle.merge([empty_o, o, empty_o], [empty_l, lse, empty_l])
    np.testing.assert_allclose(om, o, rtol=0, atol=1e-15)
    np.testing.assert_allclose(lm, lse, rtol=0, atol=1e-14)
    oz, lz = oracle.merge([empty_o, empty_o], [empty_l, empty_l])
    assert np.all(oz == 0.0) and np.all(np.isneginf(lz))


# ---------------------------------------------------------------- ring accumulate
def _ring(q, k, v, scale, bounds):
    """Ring steps over the chunks of `bounds`, from the no-key state (the
    running output holds NaN: it must not be read)."""
    B, Sq, H, D = q.shape
    o = np.full((B, Sq, H, D), np.nan)
    lse = np.full((B, H, Sq), -np.inf)
    for a, b in zip(bounds[:-1], bounds[1:]):
        o, lse = oracle.ring_accumulate(o, lse, q, np.ascontiguousarray(k[:, a:b]),
                                        np.ascontiguousarray(v[:, a:b]), scale)
    return o, lse


@pytest.mark.parametrize("bounds", [[0, 64, 128, 192, 256], [0, 1, 100, 101, 256], [0, 256]])
def test_ring_steps_equal_unchunked_attention(bounds):
    q, k, v = synth.qkv(19, 1, 2, 20, 256, 16)
    scale = F32(0.25)
    o, lse = oracle.attn(q, k, v, scale)
    orr, lr = _ring(q, k, v, scale, bounds)
    np.testing.assert_allclose(orr, o, rtol=0, atol=1e-13)
    np.testing.assert_allclose(lr, lse, rtol=0, atol=1e-12)


def test_ring_two_steps_match_brute_force_on_the_concatenated_keys():
    rng = np.random.default_rng(20)
    q, k, v = (ints_bf16(rng, s, -3, 3) for s in [(1, 3, 2, 4), (1, 7, 2, 4), (1, 7, 2, 4)])
    scale = F32(0.5)
    ob, lb = brute.attn(q, k, v, float(scale))
    orr, lr = _ring(q, k, v, scale, [0, 3, 7])
    np.testing.assert_allclose(orr, np.array(ob), rtol=0, atol=1e-13)
    np.testing.assert_allclose(lr, np.array(lb), rtol=0, atol=1e-13)


def test_ring_step_from_no_keys_is_the_chunk_result_and_ignores_the_running_output():
    q, k, v = synth.qkv(21, 1, 2, 6, 40, 8)
    scale = F32(0.3)
    o, lse = oracle.attn(q, k, v, scale)
    orr, lr = _ring(q, k, v, scale, [0, 40])
    assert np.array_equal(orr, o) and np.array_equal(lr, lse)


# ---------------------------------------------------------------- dual cross-attention
def test_dual_cross_attention_matches_two_brute_force_attentions_summed():
    rng = np.random.default_rng(22)
    q = ints_bf16(rng, (1, 4, 2, 4), -3, 3)
    kt, vt = ints_bf16(rng, (1, 5, 2, 4), -3, 3), ints_bf16(rng, (1, 5, 2, 4), -3, 3)
    ki, vi = ints_bf16(rng, (1, 3, 2, 4), -3, 3), ints_bf16(rng, (1, 3, 2, 4), -3, 3)
    scale = F32(0.5)
    o, lt, li = oracle.cross_attn_dual(q, kt, vt, ki, vi, scale)
    ot, ltb = brute.attn(q, kt, vt, float(scale))
    oi, lib = brute.attn(q, ki, vi, float(scale))
    np.testing.assert_allclose(o, np.array(ot) + np.array(oi), rtol=0, atol=1e-13)
    np.testing.assert_allclose(lt, np.array(ltb), rtol=0, atol=1e-13)
    np.testing.assert_allclose(li, np.array(lib), rtol=0, atol=1e-13)


def test_dual_cross_attention_zero_queries_give_the_two_value_means():
    """q = 0: every score is 0, each softmax is uniform over its own context:
    O = mean(V_txt) + mean(V_img), LSE = log of each context's length."""
    rng = np.random.default_rng(23)
    q = np.zeros((1, 3, 2, 8), dtype=np.uint16)
    kt, vt = synth.normal_bf16(rng, (1, 12, 2, 8)), synth.normal_bf16(rng, (1, 12, 2, 8))
    ki, vi = synth.normal_bf16(rng, (1, 5, 2, 8)), synth.normal_bf16(rng, (1, 5, 2, 8))
    o, lt, li = oracle.cross_attn_dual(q, kt, vt, ki, vi, F32(0.7))
    want = widen(vt).mean(axis=1, keepdims=True) + widen(vi).mean(axis=1, keepdims=True)
    np.testing.assert_allclose(o, np.broadcast_to(want, o.shape), rtol=0, atol=1e-14)
    assert np.allclose(lt, math.log(12), atol=1e-14) and np.allclose(li, math.log(5), atol=1e-14)


def test_dual_cross_attention_is_two_softmaxes_not_one_joint_softmax():
    """Identical contexts: the sum of two separate attentions is twice one
    attention (a joint softmax over both would return it once)."""
    q, k, v = synth.qkv(24, 1, 2, 6, 20, 8)
    o, lt, li = oracle.cross_attn_dual(q, k, v, k, v, F32(0.4))
    o1, l1 = oracle.attn(q, k, v, F32(0.4))
    np.testing.assert_allclose(o, 2.0 * o1, rtol=0, atol=1e-14)
    assert np.array_equal(lt, l1) and np.array_equal(li, l1)


# ---------------------------------------------------------------- planted mistakes
# Plausible slips in the oracle, planted in a copy of its source; each must
# make at least one pin fail.
MUTANTS = [
    ("drop the scale", "s[j] = scale * dot;", "s[j] = dot;"),
    ("wrong max sign", "const double p = exp(s[j] - m);", "const double p = exp(s[j] + m);"),
    ("unnormalized output", "oi[t] = acc[t] / l;", "oi[t] = acc[t];"),
    ("lse minus log", "lse[((int64_t)b * H + h) * Sq + i] = m + log(l);",
     "lse[((int64_t)b * H + h) * Sq + i] = m - log(l);"),
    ("lse without max", "lse[((int64_t)b * H + h) * Sq + i] = m + log(l);",
     "lse[((int64_t)b * H + h) * Sq + i] = log(l);"),
    ("key uses query stride", "k + b * k_sb + j * k_ss + h * k_sh", "k + b * k_sb + j * q_ss + h * k_sh"),
    ("value row from key", "const uint16_t *vj = v + b * v_sb", "const uint16_t *vj = k + b * v_sb"),
    ("transposed q/k index", "bf16_to_double(qi[t]) * bf16_to_double(kj[t])",
     "bf16_to_double(qi[t]) * bf16_to_double(kj[D - 1 - t])"),
    ("drop last key", "for (int j = 0; j < Skv; j++) {\n                        const double p",
     "for (int j = 0; j < Skv - 1; j++) {\n                        const double p"),
    ("merge weight sign", "const double w = exp(lse_parts[c][li] - L);",
     "const double w = exp(L - lse_parts[c][li]);"),
    ("merge lse without max", "const double L = mstar + log(sum);", "const double L = log(sum);"),
    ("merge drops a part", "for (int c = 0; c < num_parts; c++) {\n                        const double w",
     "for (int c = 1; c < num_parts; c++) {\n                        const double w"),
    ("output head index", "double *oi = o + (((int64_t)b * Sq + i) * H + h) * D;",
     "double *oi = o + (((int64_t)b * Sq + i) * H + (H - 1 - h)) * D;"),
]


def _pins_hold(lib) -> bool:
    """A compact run of the pins above against the given oracle library."""
    try:
        for (B, H, Sq, Skv, D, seed, mixed) in [(1, 2, 5, 7, 8, 1, False), (2, 2, 3, 4, 4, 4, False),
                                                (2, 3, 4, 6, 8, 5, True)]:
            q, k, v = synth.qkv(seed, B, H, Sq, Skv, D)
            if mixed:  # head-major keys, token-major queries/values: every stride differs
                k = np.ascontiguousarray(k.transpose(0, 2, 1, 3)).transpose(0, 2, 1, 3)
            scale = F32(1.0 / math.sqrt(D))
            o, lse = oracle.attn(q, k, v, scale, lib=lib)
            O, L = brute.attn(q.tolist(), k.tolist(), v.tolist(), scale)
            # written so that NaN (a mutant reading past an array) counts as a mismatch
            if not (np.abs(o - np.array(O)).max() <= 1e-12 and np.abs(lse - np.array(L)).max() <= 1e-12):
                return False
        q, k, v = synth.qkv(16, 1, 2, 6, 64, 8)
        scale = F32(0.25)
        o, lse = oracle.attn(q, k, v, scale, lib=lib)
        parts = [oracle.attn(q, np.ascontiguousarray(k[:, a:b]), np.ascontiguousarray(v[:, a:b]), scale, lib=lib)
                 for a, b in [(0, 10), (10, 40), (40, 64)]]
        om, lm = oracle.merge([p[0] for p in parts], [p[1] for p in parts], lib=lib)
        if not (np.abs(om - o).max() <= 1e-13 and np.abs(lm - lse).max() <= 1e-12):
            return False
        return True
    except Exception:
        return False


def test_planted_mistakes_are_caught():
    src = open(os.path.join(oracle.ORACLE_DIR, "oracle.c")).read()
    assert _pins_hold(oracle._load()), "the pins must hold for the real oracle"
    tmp = tempfile.mkdtemp(prefix="oracle_mutant_")
    try:
        for i, (name, old, new) in enumerate(MUTANTS):
            assert src.count(old) == 1, f"mutation site for '{name}' not found exactly once"
            # a file name no other loaded library has (the dynamic loader may
            # hand back an already loaded object it matches by name)
            path = os.path.join(tmp, f"attn_mutant_{i}.c")
            with open(path, "w") as f:
                f.write(src.replace(old, new))
            so = oracle_build.build(source=path, out=os.path.join(tmp, f"attn_mutant_{i}.so"))
            lib = oracle.open_library(so)
            assert not _pins_hold(lib), f"planted mistake '{name}' was not caught by the pins"
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
