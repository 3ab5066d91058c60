"""Host-only tests of the work plan (regenvc_attn_plan_query): the tile
decomposition an attention call of a given shape uses, and the scratch
memory it takes.  No GPU needed: the query makes no HIP call."""
import ctypes

import pytest

from paper_2607_28144_amd import _lib
from paper_2607_28144_amd.api import attn_plan

BN = 64
PAIRED_BELOW = 32  # key tiles: shorter calls run two 128-row workgroups per CU


def ceil_div(a, b):
    return -(-a // b)


def check_invariants(p, B, H, Sq, Skv, D, n_cu):
    BM = p["tile_rows"]
    assert p["key_tiles"] == ceil_div(Skv, BN)
    assert BM == (128 if p["key_tiles"] < PAIRED_BELOW else 256)
    slots = n_cu * (2 if BM == 128 else 1)  # workgroups resident at once
    assert p["query_tiles"] == B * H * ceil_div(Sq, BM)
    assert p["whole_tiles"] + p["split_tiles"] == p["query_tiles"]
    assert 0 <= p["split_tiles"] < slots
    if p["split_tiles"]:
        # only the tiles of a last, partial round over the workgroup slots are split
        assert p["whole_tiles"] % slots == 0
        assert p["whole_tiles"] == (p["query_tiles"] // slots) * slots
        assert 2 <= p["key_ranges"] <= p["key_tiles"]
    else:
        assert p["key_ranges"] == 0
    units = p["split_tiles"] * p["key_ranges"]
    assert p["workspace_bytes"] == units * BM * (D + 1) * 4


def test_window_plan():
    """12 heads x 10920 tokens (7 latent frames of 30 x 52): 516 query tiles on
    256 CUs are two full rounds plus 4 tiles, which are split along the keys."""
    p = attn_plan(1, 12, 10920, 10920, 128)
    check_invariants(p, 1, 12, 10920, 10920, 128, 256)
    assert p == {"query_tiles": 516, "key_tiles": 171, "whole_tiles": 512, "split_tiles": 4,
                 "key_ranges": 29, "workspace_bytes": 15_323_136, "tile_rows": 256}


def test_share_plan_splits_nothing():
    """One sequence-parallel rank's share, 5 heads x 10920 queries against a
    key chunk of 2730: 215 tiles fit in one round of 256 CUs."""
    p = attn_plan(1, 5, 10920, 2730, 128)
    check_invariants(p, 1, 5, 10920, 2730, 128, 256)
    assert (p["key_tiles"], p["whole_tiles"], p["split_tiles"], p["workspace_bytes"]) == (43, 215, 0, 0)


def test_cross_plan():
    """Cross-attention to 512 context tokens: 8 key tiles, so 128-row tiles
    two per CU; the 1032 tiles are two rounds of 512 plus 8, and those 8
    start only as the second round drains: each is split into 8 one-tile key
    ranges (64 units) and recombined by the fixup."""
    p = attn_plan(1, 12, 10920, 512, 128)
    check_invariants(p, 1, 12, 10920, 512, 128, 256)
    assert (p["tile_rows"], p["query_tiles"], p["key_tiles"]) == (128, 1032, 8)
    assert (p["whole_tiles"], p["split_tiles"], p["key_ranges"]) == (1024, 8, 8)
    # partials: 64 units x 128 rows x (128 O + 1 LSE) floats
    assert p["workspace_bytes"] == 64 * 128 * 129 * 4


def test_paired_leftover_tiles_after_full_rounds_split():
    """The image context (257 tokens, 5 key tiles): 1032 tiles of 128 rows
    on 512 slots, the 8 past two rounds split into 5 one-tile ranges; a
    paired launch that does not fill one round (344 tiles) keeps its tiles
    whole."""
    p = attn_plan(1, 12, 10920, 257, 128)
    check_invariants(p, 1, 12, 10920, 257, 128, 256)
    assert (p["tile_rows"], p["whole_tiles"], p["split_tiles"], p["key_ranges"]) == (128, 1024, 8, 5)
    p = attn_plan(1, 4, 10920, 512, 128)
    check_invariants(p, 1, 4, 10920, 512, 128, 256)
    assert (p["tile_rows"], p["query_tiles"], p["split_tiles"], p["workspace_bytes"]) == (128, 344, 0, 0)


def test_short_underfilled_call_splits():
    """Few 128-row tiles with many keys below the ping-pong threshold: 3
    tiles on 512 slots are split along the keys."""
    p = attn_plan(1, 1, 300, 1500, 128)
    check_invariants(p, 1, 1, 300, 1500, 128, 256)
    assert (p["tile_rows"], p["query_tiles"], p["split_tiles"]) == (128, 3, 3) and p["key_ranges"] >= 2


@pytest.mark.parametrize("B,H,Sq,Skv,D,n_cu", [
    (1, 1, 1, 1, 64, 256), (1, 1, 256, 64, 128, 1), (2, 5, 1000, 3000, 64, 7),
    (1, 12, 10920, 10920, 64, 256), (1, 12, 10920, 10920, 128, 304), (4, 24, 4096, 4096, 128, 256),
    (1, 1, 300, 65536, 128, 256), (1, 12, 10920, 10920, 128, 80),
])
def test_plan_invariants(B, H, Sq, Skv, D, n_cu):
    check_invariants(attn_plan(B, H, Sq, Skv, D, n_cu), B, H, Sq, Skv, D, n_cu)


def test_single_key_tile_is_never_split():
    p = attn_plan(1, 1, 300, 64, 128)
    assert (p["tile_rows"], p["whole_tiles"], p["split_tiles"], p["key_ranges"]) == (128, 3, 0, 0)


def test_empty_problem_plans_nothing():
    for B, H, Sq in [(0, 12, 10920), (1, 0, 10920), (1, 12, 0)]:
        p = attn_plan(B, H, Sq, 10920, 128)
        assert p["query_tiles"] == 0 and p["whole_tiles"] == 0 and p["split_tiles"] == 0
        assert p["workspace_bytes"] == 0


@pytest.mark.parametrize("args,status", [
    ((-1, 1, 1, 1, 128, 256), 1), ((1, -1, 1, 1, 128, 256), 1), ((1, 1, -1, 1, 128, 256), 1),
    ((1, 1, 1, 0, 128, 256), 1), ((1, 1, 1, 1, 128, 0), 1),
    ((1, 1, 1, 1, 96, 256), 2), ((1, 1, 1, 1, 256, 256), 2),
    ((2**31 - 1, 2**31 - 1, 2**31 - 1, 1, 128, 256), 2),
])
def test_bad_arguments_leave_the_plan_untouched(args, status):
    lib = _lib.load()
    plan = _lib.AttnPlan(query_tiles=-7, workspace_bytes=-7)
    assert lib.regenvc_attn_plan_query(*args, ctypes.byref(plan)) == status
    assert plan.query_tiles == -7 and plan.workspace_bytes == -7
    assert lib.regenvc_last_error().decode().startswith("regenvc_attn_plan_query")


def test_null_plan_is_rejected():
    lib = _lib.load()
    assert lib.regenvc_attn_plan_query(1, 1, 1, 1, 128, 256, None) == 1
