"""GPU parity of the q/k RMSNorm + 3D rotary embedding kernel (through the C
ABI) against the fp64 oracle on the same seeded bf16 inputs.

Tolerance: the kernel rounds its outputs to bf16 (nearest even: at most
half an ulp, 2^-8 relative at the bottom of a binade) and computes in
float32, where the rotation angle pos * freq carries a relative error of
~2^-23 (two roundings); the test allows
|y - y_ref| <= 2^-8 |y_ref| + (2e-6 + 4e-7 * max position) * max|y_ref|.
"""
import numpy as np
import pytest

import oracle
from paper_2607_28144_amd import synth

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

WINDOW_GRID = (7, 30, 52)  # latent frames x rows x cols of a 25-frame 480x832 window


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_28144_amd import api  # noqa: F401  (fails loudly if the library is missing)
    yield
    torch.cuda.synchronize()


def api():
    from paper_2607_28144_amd import api as a
    return a


def dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def inputs(seed, B, S, H, D):
    rng = np.random.default_rng(seed)
    q = synth.normal_bf16(rng, (B, S, H, D))
    k = synth.normal_bf16(rng, (B, S, H, D))
    wq = synth.f32_to_bf16_bits(1.0 + 0.1 * rng.standard_normal(H * D).astype(np.float32))
    wk = synth.f32_to_bf16_bits(1.0 + 0.1 * rng.standard_normal(H * D).astype(np.float32))
    return q, k, wq, wk


def check(name, y_gpu, y_ref, max_pos):
    y = y_gpu.float().cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(y)), f"{name}: non-finite output"
    err = np.abs(y - y_ref)
    bound = 2.0 ** -8 * np.abs(y_ref) + (2e-6 + 4e-7 * max_pos) * np.abs(y_ref).max()
    worst = float((err / bound).max())
    print(f"[parity] {name}: max|dy|={err.max():.3e} (max|y|={np.abs(y_ref).max():.3e}) worst err/bound={worst:.3f}",
          flush=True)
    assert worst <= 1.0, f"{name}: error exceeds the bf16 rounding bound ({worst:.3f}x)"


def run(name, seed, B, S, H, D, grid, token0=0, eps=1e-6, theta=10000.0):
    q, k, wq, wk = inputs(seed, B, S, H, D)
    qo, ko = api().qk_norm_rope(dev(q), dev(k), dev(wq), dev(wk), grid, token0=token0, eps=eps, theta=theta)
    torch.cuda.synchronize()
    max_pos = max(grid) - 1
    check(f"{name} q", qo, oracle.norm_rope(q, wq, grid, token0, eps, theta), max_pos)
    check(f"{name} k", ko, oracle.norm_rope(k, wk, grid, token0, eps, theta), max_pos)


@pytest.mark.parametrize("D", [128, 64])
def test_small_grid(D):
    run(f"small grid D={D}", 40 + D, 2, 60, 3, D, (3, 4, 5))


def test_window_shape_all_tokens():
    run("window 10920 tokens x 12 heads", 41, 1, 10920, 12, 128, WINDOW_GRID)


def test_sequence_shard_with_token_offset():
    """A contiguous shard of the window's tokens (positions continue from token0)."""
    run("window shard 5000..5999", 42, 1, 1000, 12, 128, WINDOW_GRID, token0=5000)


def test_many_heads_wide_token():
    """40 heads x 128 = 5120 channels per token (the wide-token path)."""
    run("40 heads", 43, 1, 130, 40, 128, (2, 5, 13))


def test_long_axis_positions():
    """Columns up to 4095 (the longest axis accepted): angles up to ~4095 rad."""
    run("4096 columns", 47, 1, 600, 2, 128, (1, 1, 4096), token0=3490)


def test_unit_theta_and_large_eps():
    run("theta 1, eps 0.5", 44, 1, 200, 4, 128, (2, 10, 10), eps=0.5, theta=1.0)


def test_in_place_equals_out_of_place():
    q, k, wq, wk = inputs(45, 1, 300, 12, 128)
    dq, dk = dev(q), dev(k)
    qo, ko = api().qk_norm_rope(dq, dk, dev(wq), dev(wk), (3, 10, 10))
    api().qk_norm_rope(dq, dk, dev(wq), dev(wk), (3, 10, 10), q_out=dq, k_out=dk)
    torch.cuda.synchronize()
    assert torch.equal(qo, dq) and torch.equal(ko, dk)


def test_head_major_input_layout():
    """Input stored head-major ([B,H,S,D] memory): same result bitwise."""
    q, k, wq, wk = inputs(46, 1, 120, 4, 128)
    hm = lambda x: torch.from_numpy(np.ascontiguousarray(x.transpose(0, 2, 1, 3)).view(np.int16)).view(  # noqa: E731
        torch.bfloat16).cuda().permute(0, 2, 1, 3)
    a1 = api().qk_norm_rope(dev(q), dev(k), dev(wq), dev(wk), (2, 6, 10))
    a2 = api().qk_norm_rope(hm(q), hm(k), dev(wq), dev(wk), (2, 6, 10))
    torch.cuda.synchronize()
    assert torch.equal(a1[0], a2[0]) and torch.equal(a1[1], a2[1])
