"""regenvc_attn_fwd_noalloc, the entry point for callers that cannot
allocate: the same call as regenvc_attn_fwd with its split-tile partials in
the library's static per-GPU scratch array.  Called through the C ABI and
checked against regenvc_attn_fwd's output (bitwise: same plan, same kernels;
and to the parity bar) on two calls in a row, the second with a smaller
input, while the library's pool is never drawn from; a call whose plan needs
more than the array holds is rejected before anything is enqueued.  Collected
last (the name sorts after every other test file), so that it runs both after
the rest of the suite and alone in a fresh process."""
import ctypes

import numpy as np
import pytest

from paper_2607_28144_amd import _lib, synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def desc(t):
    return _lib.Tensor(t.data_ptr(), t.stride(0), t.stride(1), t.stride(2))


def noalloc(q, k, v, o, lse, scale):
    B, Sq, H, D = q.shape
    qd, kd, vd, od = desc(q), desc(k), desc(v), desc(o)
    dt = _lib.F32 if o.dtype == torch.float32 else _lib.BF16
    return _lib.load().regenvc_attn_fwd_noalloc(ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd),
                                                ctypes.byref(od), dt, lse.data_ptr(), B, H, Sq, k.shape[1], D,
                                                scale, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))


def need(B, H, Sq, Skv, D):
    from paper_2607_28144_amd import api
    return api.attn_plan(B, H, Sq, Skv, D, torch.cuda.get_device_properties(0).multi_processor_count)[
        "workspace_bytes"]


def test_noalloc_matches_attn_fwd_on_two_calls_in_a_row():
    from paper_2607_28144_amd import api
    cases = [(3, 1, 12, 10920, 10920, 128, torch.bfloat16),  # the window: 14.6 MiB of scratch
             (41, 1, 4, 3000, 3000, 128, torch.float32)]     # a smaller input, every tile split: 24.2 MiB
    for seed, B, H, Sq, Skv, D, dt in cases:
        assert 0 < need(B, H, Sq, Skv, D) <= 32 << 20
        q, k, v = (dev(x) for x in synth.qkv(seed, B, H, Sq, Skv, D))
        scale = synth.default_scale(D)
        o_ref, l_ref = api.attn_fwd(q, k, v, scale=scale, out_dtype=dt)
        o = torch.full_like(o_ref, float("nan"))
        lse = torch.full_like(l_ref, float("nan"))
        draws = api.pool_draws()
        print(f"[no-alloc] B={B} H={H} Sq={Sq} Skv={Skv} D={D} scratch={need(B, H, Sq, Skv, D)} bytes", flush=True)
        assert noalloc(q, k, v, o, lse, scale) == _lib.OK, _lib.load().regenvc_last_error()
        torch.cuda.synchronize()
        assert api.pool_draws() == draws
        d_o = (o.float() - o_ref.float()).abs().max().item()
        d_l = (lse - l_ref).abs().max().item()
        print(f"[no-alloc] vs regenvc_attn_fwd: max|dO|={d_o:.3e} max|dLSE|={d_l:.3e}", flush=True)
        assert d_o <= 1e-2 and d_o <= 1e-2 * o_ref.float().abs().max().item() and d_l <= 1e-3
        assert torch.equal(o, o_ref) and torch.equal(lse, l_ref)


def test_noalloc_rejects_a_plan_beyond_its_scratch():
    from paper_2607_28144_amd import api
    B, H, Sq, Skv, D = 1, 2, 4000, 8000, 128
    assert need(B, H, Sq, Skv, D) > 32 << 20
    q, k, v = (dev(x) for x in synth.qkv(42, B, H, Sq, Skv, D))
    o = torch.full((B, Sq, H, D), 3.0, dtype=torch.bfloat16, device="cuda")
    lse = torch.full((B, H, Sq), 3.0, dtype=torch.float32, device="cuda")
    draws = api.pool_draws()
    st = noalloc(q, k, v, o, lse, synth.default_scale(D))
    torch.cuda.synchronize()
    assert st == _lib.ERR_UNSUPPORTED and b"more than" in _lib.load().regenvc_last_error()
    assert api.pool_draws() == draws
    assert torch.all(o == 3.0) and torch.all(lse == 3.0)
