"""GPU parity of the ring accumulate (regenvc_attn_ring_accumulate): partial
attention over one key/value chunk whose epilogue merges the result into the
running (O, LSE) state, against the oracle's ring step (fp64) on the same
seeded bf16 inputs.  Tolerances as for the other attention entry points:
max |dO| <= 1e-2 (and <= 1e-2 * max|O|), max |dLSE| <= 1e-3."""
import numpy as np
import pytest

import oracle
from paper_2607_28144_amd import synth
from test_gpu_parity import api, assert_close, dev, host, sample_rows

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def _chunk(x, a, b):
    return np.ascontiguousarray(x[:, a:b])


def _ring_check(name, q, k, v, bounds, rows=None, fresh=True, final_bf16=True):
    """Runs the ring over the chunks of `bounds` on the GPU and checks the
    running state after every step against the oracle's ring steps (on the
    query rows `rows`, or all).  fresh: start from lse = -inf with a running
    output full of NaN (it must not be read); else start with a partial of
    the first chunk.  final_bf16: the last step writes a separate bf16
    output."""
    B, Sq, H, D = q.shape
    scale = synth.default_scale(D)
    dq, dk, dv = dev(q), dev(k), dev(v)
    qs = q if rows is None else np.ascontiguousarray(q[:, rows])
    pick_o = (lambda t: host(t)) if rows is None else (lambda t: host(t)[:, rows])
    pick_l = (lambda t: t.cpu().numpy()) if rows is None else (lambda t: t.cpu().numpy()[:, :, rows])
    steps = list(zip(bounds[:-1], bounds[1:]))
    if fresh:
        o_run = torch.full((B, Sq, H, D), float("nan"), dtype=torch.float32, device="cuda")
        lse_run = torch.full((B, H, Sq), float("-inf"), dtype=torch.float32, device="cuda")
        o_ref = np.full((B, qs.shape[1], H, D), np.nan)
        l_ref = np.full((B, H, qs.shape[1]), -np.inf)
    else:
        a, b = steps.pop(0)
        o_run, lse_run = api().attn_partial_fwd(dq, dk[:, a:b], dv[:, a:b], scale=scale)
        o_ref, l_ref = oracle.attn(qs, _chunk(k, a, b), _chunk(v, a, b), scale)
    for i, (a, b) in enumerate(steps):
        last = i == len(steps) - 1
        if last and final_bf16:
            res = api().attn_ring_accumulate(dq, dk[:, a:b], dv[:, a:b], o_run, lse_run, scale=scale,
                                             out=torch.empty((B, Sq, H, D), dtype=torch.bfloat16, device="cuda"),
                                             out_dtype=torch.bfloat16)
        else:
            res = api().attn_ring_accumulate(dq, dk[:, a:b], dv[:, a:b], o_run, lse_run, scale=scale)
            assert res.data_ptr() == o_run.data_ptr()
        torch.cuda.synchronize()
        o_ref, l_ref = oracle.ring_accumulate(o_ref, l_ref, qs, _chunk(k, a, b), _chunk(v, a, b), scale)
        assert_close(f"{name} step {i} keys {a}..{b}", pick_o(res), o_ref, pick_l(lse_run), l_ref)
    return res, lse_run


def test_ring_rank_share_config():
    """H=5 heads, Sq=10920, keys in 4 chunks of 2730: the first chunk's
    partial, two in-place steps, and a last step into bf16 (sampled rows)."""
    B, H, S, D = 1, 5, 10920, 128
    q, k, v = synth.qkv(4, B, H, S, S, D)
    res, lse = _ring_check("ring share", q, k, v, [0, 2730, 5460, 8190, 10920], rows=sample_rows(S, 48, 4),
                           fresh=False)
    # the ring equals partials + merge on the same device up to fp32 rounding
    dq, dk, dv = dev(q), dev(k), dev(v)
    scale = synth.default_scale(D)
    parts = [api().attn_partial_fwd(dq, dk[:, a:b], dv[:, a:b], scale=scale)
             for a, b in [(0, 2730), (2730, 5460), (5460, 8190), (8190, 10920)]]
    om, lm = api().lse_merge([p[0] for p in parts], [p[1] for p in parts], out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    d_o = (om.float() - res.float()).abs().max().item()
    d_l = (lm - lse).abs().max().item()
    print(f"[parity] ring vs partials + merge: max|dO|={d_o:.3e} max|dLSE|={d_l:.3e}", flush=True)
    assert d_o <= 2 ** -7 and d_l <= 1e-5


@pytest.mark.parametrize("schedule", ["interleaved", "pingpong", "paired"])
@pytest.mark.parametrize("bounds", [[0, 1, 100, 101, 777], [0, 640, 777]])
def test_ring_ragged_chunks_from_no_keys(schedule, bounds, monkeypatch):
    """Uneven and single-token chunks, 300 queries (a ragged query tile),
    starting from the no-key state whose running output is NaN."""
    monkeypatch.setenv("REGENVC_ATTN_SCHEDULE", schedule)
    q, k, v = synth.qkv(50 + len(bounds), 2, 2, 300, 777, 128)
    _ring_check(f"ring {schedule} {bounds}", q, k, v, bounds)


def test_ring_head_dim_64_f32_final_output():
    q, k, v = synth.qkv(55, 1, 3, 200, 500, 64)
    _ring_check("ring D=64", q, k, v, [0, 250, 500], final_bf16=False)


def test_ring_split_tiles_go_through_the_fixup():
    """12 heads x 10920 queries: 516 query tiles on 256 CUs, so the plan
    splits the last tiles along the keys and their fixup kernel does the
    merge into the running state; every row of those tiles is checked."""
    B, H, S, D = 1, 12, 10920, 128
    plan = api().attn_plan(B, H, S, 2730, D)
    assert plan["split_tiles"] > 0, plan
    q, k, v = synth.qkv(3, B, H, S, S, D)
    first_split_row = S - plan["split_tiles"] * 256 + (-S) % 256
    rows = np.unique(np.concatenate([np.arange(max(first_split_row - 64, 0), S), sample_rows(S, 16, 7)]))
    hq = np.ascontiguousarray(q[:, :, 11:12])  # the split tiles are the last ones: the last head
    hk, hv = np.ascontiguousarray(k[:, :, 11:12]), np.ascontiguousarray(v[:, :, 11:12])
    scale = synth.default_scale(D)
    dq, dk, dv = dev(q), dev(k), dev(v)
    o_run, lse_run = api().attn_partial_fwd(dq, dk[:, :2730], dv[:, :2730], scale=scale)
    out = api().attn_ring_accumulate(dq, dk[:, 2730:5460], dv[:, 2730:5460], o_run, lse_run, scale=scale,
                                     out=torch.empty((B, S, H, D), dtype=torch.bfloat16, device="cuda"),
                                     out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    qs = np.ascontiguousarray(hq[:, rows])
    o_ref, l_ref = oracle.attn(qs, _chunk(hk, 0, 5460), _chunk(hv, 0, 5460), scale)
    assert_close("ring split tiles head 11", host(out)[:, rows][:, :, 11:12], o_ref,
                 lse_run.cpu().numpy()[:, 11:12][:, :, rows], l_ref)


def test_ring_step_into_a_separate_f32_output_leaves_the_running_output():
    """o_out given in f32: the merged output goes there, o_run is only read
    (unchanged), and lse_run is updated in place."""
    q, k, v = synth.qkv(56, 1, 2, 300, 600, 128)
    scale = synth.default_scale(128)
    dq, dk, dv = dev(q), dev(k), dev(v)
    o_run, lse_run = api().attn_partial_fwd(dq, dk[:, :250], dv[:, :250], scale=scale)
    before = o_run.clone()
    out = torch.empty_like(o_run)
    res = api().attn_ring_accumulate(dq, dk[:, 250:], dv[:, 250:], o_run, lse_run, scale=scale, out=out,
                                     out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert res.data_ptr() == out.data_ptr()
    assert torch.equal(o_run, before)
    o_ref, l_ref = oracle.attn(q, k, v, scale)
    assert_close("ring step into a separate f32 output", out, o_ref, lse_run, l_ref)
