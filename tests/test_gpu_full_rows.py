"""Every query row of each configuration at full size, against the fp64
oracle on the host cores, through the C ABI.

One test per configuration, in the launch configuration the benchmark times:
  image   B=1, H=12, S=4096, d=128, bf16 O + LSE                 (seed 2)
  window  B=1, H=12, S=10920 = 7 x 30 x 52, d=128, bf16 O + LSE  (seed 3)
  cross   the window's 10920 queries to 512 context tokens        (seed 3)
  share   H=5, Sq=10920, keys in 4 chunks of 2730: each chunk's f32
          partial, the LSE merge into bf16, and the same share through
          ring-accumulate steps                                   (seed 4)
  paper   H=3, Sq=5460, keys in 2 chunks of 5460: partials + merge (seed 5)
Each comparison prints max-abs, RMS and normalized errors and the count of
elements over tolerance (tests/test_gpu_parity.py: max|dO| <= 1e-2 and
<= 1e-2 * max|O|, max|dLSE| <= 1e-3) and asserts the bar on all rows.
"""
import functools

import numpy as np
import pytest

import oracle
from paper_2607_28144_amd import synth
from test_gpu_parity import api, assert_close, dev, host

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

WINDOW = dict(B=1, H=12, S=10920, D=128, seed=3, ctx=512)
SHARE = dict(B=1, H=5, S=10920, D=128, seed=4, bounds=(0, 2730, 5460, 8190, 10920))
PAPER = dict(B=1, H=3, S=10920, Sq=5460, D=128, seed=5, bounds=(0, 5460, 10920))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


@functools.lru_cache(maxsize=None)
def window_inputs():
    W = WINDOW
    return synth.qkv(W["seed"], W["B"], W["H"], W["S"], W["S"], W["D"], ctx=W["ctx"])


@functools.lru_cache(maxsize=None)
def share_inputs():
    R = SHARE
    return synth.qkv(R["seed"], R["B"], R["H"], R["S"], R["S"], R["D"])


@functools.lru_cache(maxsize=None)
def share_reference():
    q, k, v = share_inputs()
    return oracle.attn(q, k, v, synth.default_scale(SHARE["D"]))


def lse_host(t):
    return t.cpu().numpy().astype(np.float64)


def test_image_config_every_row():
    B, H, S, D = 1, 12, 4096, 128
    q, k, v = synth.qkv(2, B, H, S, S, D)
    scale = synth.default_scale(D)
    o, lse = api().attn_fwd(dev(q), dev(k), dev(v), scale=scale)
    torch.cuda.synchronize()
    o_ref, l_ref = oracle.attn(q, k, v, scale)
    assert_close("image S=4096 H=12 every row", o, o_ref, lse, l_ref)


def test_window_self_attention_every_row():
    W = WINDOW
    q, k, v, _, _ = window_inputs()
    scale = synth.default_scale(W["D"])
    o, lse = api().attn_fwd(dev(q), dev(k), dev(v), scale=scale)
    torch.cuda.synchronize()
    o_ref, l_ref = oracle.attn(q, k, v, scale)
    assert_close("window self S=10920 H=12 every row", o, o_ref, lse, l_ref)


def test_window_cross_attention_every_row():
    W = WINDOW
    q, _, _, kc, vc = window_inputs()
    scale = synth.default_scale(W["D"])
    o, lse = api().cross_attn_fwd(dev(q), dev(kc), dev(vc), scale=scale)
    torch.cuda.synchronize()
    o_ref, l_ref = oracle.attn(q, kc, vc, scale)
    assert_close("window cross 10920 -> 512 every row", o, o_ref, lse, l_ref)


def test_rank_share_partials_and_merge_every_row():
    R = SHARE
    q, k, v = share_inputs()
    scale = synth.default_scale(R["D"])
    b = R["bounds"]
    dq, dk, dv = dev(q), dev(k), dev(v)
    parts = [api().attn_partial_fwd(dq, dk[:, a:c], dv[:, a:c], scale=scale) for a, c in zip(b[:-1], b[1:])]
    o, lse = api().lse_merge([p[0] for p in parts], [p[1] for p in parts], out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    for i, (a, c) in enumerate(zip(b[:-1], b[1:])):
        o_ref, l_ref = oracle.attn(q, np.ascontiguousarray(k[:, a:c]), np.ascontiguousarray(v[:, a:c]), scale)
        assert_close(f"share chunk {i} keys {a}..{c - 1} every row", parts[i][0], o_ref, parts[i][1], l_ref)
    o_ref, l_ref = share_reference()
    assert_close("share merged (bf16) every row", o, o_ref, lse, l_ref)


def test_rank_share_ring_steps_every_row():
    """The share through ring steps: the first chunk's partial, then three
    ring-accumulate steps, the last into bf16."""
    R = SHARE
    q, k, v = share_inputs()
    scale = synth.default_scale(R["D"])
    b = R["bounds"]
    dq, dk, dv = dev(q), dev(k), dev(v)
    o_run, l_run = api().attn_partial_fwd(dq, dk[:, b[0]:b[1]], dv[:, b[0]:b[1]], scale=scale)
    out = torch.empty(q.shape, dtype=torch.bfloat16, device="cuda")
    for i in range(1, len(b) - 1):
        last = i == len(b) - 2
        api().attn_ring_accumulate(dq, dk[:, b[i]:b[i + 1]], dv[:, b[i]:b[i + 1]], o_run, l_run, scale=scale,
                                   out=out if last else None, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    o_ref, l_ref = share_reference()
    assert_close("share ring steps (bf16) every row", out, o_ref, l_run, l_ref)


def test_paper_share_every_row():
    P = PAPER
    q, k, v = synth.qkv(P["seed"], P["B"], P["H"], P["S"], P["S"], P["D"])
    q = np.ascontiguousarray(q[:, :P["Sq"]])
    scale = synth.default_scale(P["D"])
    b = P["bounds"]
    dq, dk, dv = dev(q), dev(k), dev(v)
    parts = [api().attn_partial_fwd(dq, dk[:, a:c], dv[:, a:c], scale=scale) for a, c in zip(b[:-1], b[1:])]
    o, lse = api().lse_merge([p[0] for p in parts], [p[1] for p in parts])
    torch.cuda.synchronize()
    o_ref, l_ref = oracle.attn(q, k, v, scale)
    assert_close("paper share H=3 Sq=5460 every row", o, o_ref, lse, l_ref)
