"""GPU parity of the chunked partials (regenvc_attn_partials_fwd): every
chunk's partial of one launch against the fp64 oracle on that chunk's keys,
against the per-chunk regenvc_attn_partial_fwd results, and merged
(regenvc_lse_merge) against the oracle over all keys.  Same bar as the other
attention tests (tests/test_gpu_parity.py): max |dO| <= 1e-2 and
<= 1e-2 max|O|, max |dLSE| <= 1e-3.
"""
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
    from paper_2607_28144_amd import api as _  # noqa: F401  (fails loudly if the library is missing)
    yield
    torch.cuda.synchronize()


def per_chunk(dq, dk, dv, bounds, scale):
    return [api().attn_partial_fwd(dq, dk[:, a:b], dv[:, a:b], scale=scale) for a, b in zip(bounds[:-1], bounds[1:])]


def check_against_oracle(name, q, k, v, bounds, scale, outs, lses, rows=None):
    qs = q if rows is None else np.ascontiguousarray(q[:, rows])
    for c, (a, b) in enumerate(zip(bounds[:-1], bounds[1:])):
        o_ref, l_ref = oracle.attn(qs, np.ascontiguousarray(k[:, a:b]), np.ascontiguousarray(v[:, a:b]), scale)
        og, lg = host(outs[c]), lses[c].cpu().numpy()
        if rows is not None:
            og, lg = og[:, rows], lg[:, :, rows]
        assert_close(f"{name} chunk {c} [{a}, {b})", og, o_ref, lg, l_ref)


def test_rank_share_chunks_in_one_launch():
    """The rank share (H=5, Sq=10920, 4 chunks of 2730) in one launch: 860
    query tiles, the last 92 split along the keys.  The tiles both launches
    keep whole are bitwise equal to the per-chunk partials; the split ones
    agree within rounding; the merge matches the oracle (sampled rows, and
    every row of the split tiles' sample) and the unchunked kernel."""
    B, H, S, D = 1, 5, 10920, 128
    q, k, v = synth.qkv(4, B, H, S, S, D)
    scale = synth.default_scale(D)
    bounds = [0, 2730, 5460, 8190, 10920]
    dq, dk, dv = dev(q), dev(k), dev(v)
    plan = api().attn_plan(B, H, S, 2730, D)  # per-chunk launches keep all 215 tiles whole
    assert plan["split_tiles"] == 0
    outs, lses = api().attn_partials_fwd(dq, dk, dv, bounds, scale=scale)
    ref = per_chunk(dq, dk, dv, bounds, scale)
    torch.cuda.synchronize()
    # tiles of the chunked launch: chunk c, head h, query tile t -> index (c * H + h) * 43 + t; the last 92 are split
    n_qt = (S + 255) // 256
    first_split = 4 * H * n_qt - 92
    for c in range(4):
        for h in range(H):
            split_from = min(max(first_split - (c * H + h) * n_qt, 0), n_qt) * 256
            whole = slice(0, min(split_from, S))
            if whole.stop > 0:
                assert torch.equal(outs[c][:, whole, h], ref[c][0][:, whole, h]), (c, h)
                assert torch.equal(lses[c][:, h, whole], ref[c][1][:, h, whole]), (c, h)
            if split_from < S:
                d_o = (outs[c][:, split_from:, h] - ref[c][0][:, split_from:, h]).abs().max().item()
                d_l = (lses[c][:, h, split_from:] - ref[c][1][:, h, split_from:]).abs().max().item()
                print(f"[partials] chunk {c} head {h} split rows from {split_from}: max|dO|={d_o:.3e} "
                      f"max|dLSE|={d_l:.3e} against the per-chunk launch", flush=True)
                # each key range rounds its weights to bf16 against its own reference
                o_max = ref[c][0][:, split_from:, h].abs().max().item()
                assert d_o <= 1e-2 * o_max and d_l <= 1e-3
    rows = sample_rows(S, 48, 41)
    check_against_oracle("rank share, one launch", q, k, v, bounds, scale, outs, lses, rows)
    # rows inside the split tiles of the last chunk (heads 2-4)
    split_rows = np.array(sorted({9472, 9473, 9727, 9728, 10000, 10500, 10918, 10919}))
    check_against_oracle("rank share, split tiles", q, k, v, bounds, scale, outs, lses, split_rows)
    o, lse = api().lse_merge(outs, lses, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    o_ref, l_ref = oracle.attn(np.ascontiguousarray(q[:, rows]), k, v, scale)
    assert_close("rank share merged (one launch)", host(o)[:, rows], o_ref, lse.cpu().numpy()[:, :, rows], l_ref)
    o_full, l_full = api().attn_fwd(dq, dk, dv, scale=scale, out_dtype=torch.float32)
    o32, l32 = api().lse_merge(outs, lses, out_dtype=torch.float32)
    torch.cuda.synchronize()
    d_o, d_l = (o_full - o32).abs().max().item(), (l_full - l32).abs().max().item()
    print(f"[partials] merged one-launch partials vs unchunked kernel: max|dO|={d_o:.3e} max|dLSE|={d_l:.3e}",
          flush=True)
    assert d_o <= 1e-3 and d_l <= 1e-4


@pytest.mark.parametrize("B,H,Sq,bounds,Skv", [
    (2, 3, 700, [5, 69, 70, 400, 777], 777),    # chunks of 1 to 6 key tiles, the first not at 0: nothing split
    (1, 2, 1000, [0, 3000, 6000, 9000], 9100),  # 24 tiles on 256 CUs: every tile split, keys beyond the last chunk
    (1, 1, 300, [0, 64, 128, 129, 1000], 1000),  # whole-tile and one-key chunks, a ragged query tile
])
def test_uneven_chunks_every_row(B, H, Sq, bounds, Skv):
    D = 128
    q, k, v = synth.qkv(43, B, H, Sq, Skv, D)
    scale = synth.default_scale(D)
    dq, dk, dv = dev(q), dev(k), dev(v)
    outs, lses = api().attn_partials_fwd(dq, dk, dv, bounds, scale=scale)
    torch.cuda.synchronize()
    check_against_oracle(f"chunks {bounds}", q, k, v, bounds, scale, outs, lses)
    o, lse = api().lse_merge(outs, lses, out_dtype=torch.float32)
    torch.cuda.synchronize()
    a, b = bounds[0], bounds[-1]
    o_ref, l_ref = oracle.attn(q, np.ascontiguousarray(k[:, a:b]), np.ascontiguousarray(v[:, a:b]), scale)
    assert_close(f"chunks {bounds} merged", o, o_ref, lse, l_ref)


def test_one_chunk_is_the_plain_partial_bitwise():
    """num_chunks = 1 on keys [100, 2830) gives exactly the partial of that view."""
    B, H, S, D = 1, 5, 10920, 128
    q, k, v = synth.qkv(44, B, H, 2000, S, D)
    scale = synth.default_scale(D)
    dq, dk, dv = dev(q), dev(k), dev(v)
    outs, lses = api().attn_partials_fwd(dq, dk, dv, [100, 2830], scale=scale)
    o1, l1 = api().attn_partial_fwd(dq, dk[:, 100:2830], dv[:, 100:2830], scale=scale)
    torch.cuda.synchronize()
    assert torch.equal(outs[0], o1) and torch.equal(lses[0], l1)


def test_paper_share_chunks_in_one_launch():
    """The paper's own share (H=3, 5460 queries, 2 chunks of 5460) in one
    launch, merged, against the oracle on sampled rows."""
    B, H, S, D = 1, 3, 10920, 128
    q, k, v = synth.qkv(5, B, H, S, S, D)
    q = np.ascontiguousarray(q[:, :5460])
    scale = synth.default_scale(D)
    bounds = [0, 5460, 10920]
    dq, dk, dv = dev(q), dev(k), dev(v)
    outs, lses = api().attn_partials_fwd(dq, dk, dv, bounds, scale=scale)
    o, lse = api().lse_merge(outs, lses)
    torch.cuda.synchronize()
    rows = sample_rows(5460, 48, 45)
    check_against_oracle("paper share, one launch", q, k, v, bounds, scale, outs, lses, rows)
    o_ref, l_ref = oracle.attn(np.ascontiguousarray(q[:, rows]), k, v, scale)
    assert_close("paper share merged (one launch)", host(o)[:, rows], o_ref, lse.cpu().numpy()[:, :, rows], l_ref)
