"""Host-side tests of the C ABI (include/regenvc_attn.h): the library loads,
exports every declared entry point, and rejects bad arguments synchronously,
before any HIP call.  The fake device addresses used here are never
dereferenced: every case fails validation (or is an empty problem) first."""
import ctypes
import os
import re

import pytest

from conftest import REPO, has_gpu_node
from paper_2607_28144_amd import _lib

HEADER = os.path.join(REPO, "include", "regenvc_attn.h")
FAKE = 0x10000000  # 16-byte aligned, never dereferenced


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def declared_functions():
    text = "".join(open(os.path.join(REPO, "include", h)).read()
                   for h in ("regenvc_attn.h", "regenvc_dit.h", "regenvc_vae.h"))
    return sorted(set(re.findall(r"^\s*(?:regenvc_status|const char \*|int64_t)\s*(regenvc_\w+)\s*\(", text, re.M)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ["regenvc_attn_fwd", "regenvc_attn_partial_fwd", "regenvc_lse_merge", "regenvc_cross_attn_fwd",
              "regenvc_status_str", "regenvc_last_error", "regenvc_attn_set_workspace",
              "regenvc_cross_attn_dual_plan_query", "regenvc_attn_pool_draws"]:
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), f"{name} declared in the header but not exported"


def test_status_strings(lib):
    assert lib.regenvc_status_str(0) == b"ok"
    assert b"invalid" in lib.regenvc_status_str(1)
    assert lib.regenvc_status_str(2) == b"unsupported"
    assert b"HIP" in lib.regenvc_status_str(3)


def T(ptr=FAKE, sb=None, ss=None, sh=None, S=64, H=2, D=128):
    """Token-major [B,S,H,D] descriptor at a fake address."""
    return _lib.Tensor(ptr, S * H * D if sb is None else sb, H * D if ss is None else ss, D if sh is None else sh)


def attn(lib, q=None, k=None, v=None, o=None, dtype=_lib.BF16, lse=None, B=1, H=2, Sq=64, Skv=64, D=128,
         scale=0.088, fn="regenvc_attn_fwd"):
    q = q if q is not None else T(FAKE, S=Sq, H=H, D=D)
    k = k if k is not None else T(FAKE + 0x1000000, S=Skv, H=H, D=D)
    v = v if v is not None else T(FAKE + 0x2000000, S=Skv, H=H, D=D)
    o = o if o is not None else T(FAKE + 0x3000000, S=Sq, H=H, D=D)
    byref = lambda t: ctypes.byref(t) if t is not False else None  # noqa: E731
    if fn == "regenvc_attn_partial_fwd":
        return lib.regenvc_attn_partial_fwd(byref(q), byref(k), byref(v), byref(o), lse, B, H, Sq, Skv, D,
                                            scale, None)
    return getattr(lib, fn)(byref(q), byref(k), byref(v), byref(o), dtype, lse, B, H, Sq, Skv, D, scale, None)


def expect(lib, status, want, fragment=None):
    assert status == want, (status, lib.regenvc_last_error())
    if want != _lib.OK and fragment is not None:
        assert fragment in lib.regenvc_last_error().decode(), lib.regenvc_last_error()


@pytest.mark.parametrize("fn", ["regenvc_attn_fwd", "regenvc_cross_attn_fwd", "regenvc_attn_partial_fwd"])
def test_invalid_arguments_are_rejected_before_any_launch(lib, fn):
    LSE = FAKE + 0x4000000
    kw = dict(fn=fn, lse=LSE if fn == "regenvc_attn_partial_fwd" else None)
    expect(lib, attn(lib, q=False, **kw), _lib.ERR_INVALID_ARG, "NULL")
    expect(lib, attn(lib, q=T(0), **kw), _lib.ERR_INVALID_ARG, "NULL")
    expect(lib, attn(lib, B=-1, **kw), _lib.ERR_INVALID_ARG, "negative")
    expect(lib, attn(lib, Sq=-5, **kw), _lib.ERR_INVALID_ARG, "negative")
    expect(lib, attn(lib, Skv=-1, **kw), _lib.ERR_INVALID_ARG, "key count")
    expect(lib, attn(lib, D=96, **kw), _lib.ERR_UNSUPPORTED, "head dim")
    expect(lib, attn(lib, D=256, **kw), _lib.ERR_UNSUPPORTED, "head dim")
    expect(lib, attn(lib, scale=float("nan"), **kw), _lib.ERR_INVALID_ARG, "finite")
    expect(lib, attn(lib, scale=float("inf"), **kw), _lib.ERR_INVALID_ARG, "finite")
    expect(lib, attn(lib, scale=-0.5, **kw), _lib.ERR_INVALID_ARG, "negative")
    expect(lib, attn(lib, q=T(FAKE + 8), **kw), _lib.ERR_UNSUPPORTED, "aligned")
    expect(lib, attn(lib, k=T(FAKE + 0x1000000, ss=260), **kw), _lib.ERR_UNSUPPORTED, "multiple of 8")
    expect(lib, attn(lib, o=T(FAKE), **kw), _lib.ERR_INVALID_ARG, "overlaps")  # o on top of q
    expect(lib, attn(lib, o=T(FAKE + 0x3000000, ss=0), **kw), _lib.ERR_INVALID_ARG, "overlapping rows")
    expect(lib, attn(lib, o=T(FAKE + 0x3000000, sb=0, ss=128, sh=64), B=1, **kw), _lib.ERR_INVALID_ARG,
           "overlapping rows")  # heads interleaved into one another
    expect(lib, attn(lib, k=T(FAKE + 0x1000000, ss=-(2 ** 62)), Skv=64, **kw), _lib.ERR_UNSUPPORTED, "overflow")
    if fn != "regenvc_attn_partial_fwd":
        expect(lib, attn(lib, Skv=0, **kw), _lib.ERR_INVALID_ARG, "key count")
        expect(lib, attn(lib, dtype=7, **kw), _lib.ERR_INVALID_ARG, "dtype")
        expect(lib, attn(lib, lse=FAKE + 0x3000000 + 4, fn=fn), _lib.ERR_INVALID_ARG, "lse overlaps")
        expect(lib, attn(lib, lse=FAKE + 0x4000002, fn=fn), _lib.ERR_UNSUPPORTED, "aligned")
    else:
        expect(lib, attn(lib, fn=fn, lse=None), _lib.ERR_INVALID_ARG, "required")


@pytest.mark.parametrize("fn", ["regenvc_attn_fwd", "regenvc_cross_attn_fwd", "regenvc_attn_partial_fwd"])
def test_empty_problems_succeed_without_touching_memory(lib, fn):
    LSE = FAKE + 0x4000000
    for B, H, Sq in [(0, 2, 64), (1, 0, 64), (1, 2, 0)]:
        expect(lib, attn(lib, B=B, H=H, Sq=Sq, fn=fn, lse=LSE), _lib.OK)
    assert lib.regenvc_last_error() == b""


def merge(lib, n=2, o=None, lse=None, parts=None, lparts=None, dtype=_lib.BF16, B=1, H=2, Sq=64, D=128):
    o = o if o is not None else T(FAKE + 0x3000000, S=Sq, H=H, D=D)
    size = B * Sq * H * D * 4
    parts = parts if parts is not None else [FAKE + 0x5000000 + i * 0x1000000 for i in range(max(n, 0))]
    lparts = lparts if lparts is not None else [FAKE + 0x20000000 + i * 0x100000 for i in range(max(n, 0))]
    assert size < 0x1000000
    pa = (ctypes.c_void_p * max(len(parts), 1))(*parts)
    la = (ctypes.c_void_p * max(len(lparts), 1))(*lparts)
    return lib.regenvc_lse_merge(pa, la, n, ctypes.byref(o), dtype, lse, B, H, Sq, D, None)


def test_merge_validation(lib):
    expect(lib, merge(lib, n=0), _lib.ERR_INVALID_ARG, "num_parts")
    expect(lib, merge(lib, n=17, parts=[FAKE] * 17, lparts=[FAKE] * 17), _lib.ERR_INVALID_ARG, "num_parts")
    expect(lib, merge(lib, parts=[FAKE + 0x5000000, 0]), _lib.ERR_INVALID_ARG, "NULL")
    expect(lib, merge(lib, parts=[FAKE + 0x5000008, FAKE + 0x6000000]), _lib.ERR_UNSUPPORTED, "aligned")
    expect(lib, merge(lib, D=32), _lib.ERR_UNSUPPORTED, "head dim")
    expect(lib, merge(lib, dtype=3), _lib.ERR_INVALID_ARG, "dtype")
    expect(lib, merge(lib, o=T(FAKE + 0x5000000)), _lib.ERR_INVALID_ARG, "overlaps part")
    expect(lib, merge(lib, lse=FAKE + 0x20000000), _lib.ERR_INVALID_ARG, "overlaps part")
    expect(lib, merge(lib, o=T(FAKE + 0x3000000, ss=0)), _lib.ERR_INVALID_ARG, "overlapping rows")
    expect(lib, merge(lib, B=0), _lib.OK)


@pytest.mark.skipif(has_gpu_node(), reason="would reach a launch on fake addresses on a GPU machine")
def test_valid_arguments_without_a_gpu_report_a_hip_error(lib):
    # Validation passes, then the device query fails: nothing can be launched.
    expect(lib, attn(lib), _lib.ERR_HIP, "hip")


def norm_rope(lib, q=None, k=None, qo=None, ko=None, wq=FAKE + 0x6000000, wk=FAKE + 0x6100000, B=1, S=64, H=2,
              D=128, grid=(4, 4, 4), token0=0, eps=1e-6, theta=10000.0):
    q = q if q is not None else T(FAKE, S=S, H=H, D=D)
    k = k if k is not None else T(FAKE + 0x1000000, S=S, H=H, D=D)
    qo = qo if qo is not None else T(FAKE + 0x2000000, S=S, H=H, D=D)
    ko = ko if ko is not None else T(FAKE + 0x3000000, S=S, H=H, D=D)
    byref = lambda t: ctypes.byref(t) if t is not False else None  # noqa: E731
    return lib.regenvc_qk_norm_rope(byref(q), byref(k), wq, wk, byref(qo), byref(ko), B, S, H, D, *grid, token0,
                                    eps, theta, None)


def test_norm_rope_validation(lib):
    expect(lib, norm_rope(lib, D=96), _lib.ERR_UNSUPPORTED, "head dim")
    expect(lib, norm_rope(lib, H=0), _lib.ERR_INVALID_ARG, "bad size")
    expect(lib, norm_rope(lib, H=65, D=128), _lib.ERR_UNSUPPORTED, "channels")
    expect(lib, norm_rope(lib, grid=(4, 4, 3)), _lib.ERR_INVALID_ARG, "outside")
    expect(lib, norm_rope(lib, token0=1), _lib.ERR_INVALID_ARG, "outside")
    expect(lib, norm_rope(lib, grid=(0, 4, 4)), _lib.ERR_INVALID_ARG, "grid")
    expect(lib, norm_rope(lib, grid=(1, 1, 4097)), _lib.ERR_UNSUPPORTED, "longer than 4096")
    expect(lib, norm_rope(lib, eps=-1.0), _lib.ERR_INVALID_ARG, "eps")
    expect(lib, norm_rope(lib, eps=float("nan")), _lib.ERR_INVALID_ARG, "eps")
    expect(lib, norm_rope(lib, theta=0.0), _lib.ERR_INVALID_ARG, "theta")
    expect(lib, norm_rope(lib, wq=0), _lib.ERR_INVALID_ARG, "weight")
    expect(lib, norm_rope(lib, wk=FAKE + 8), _lib.ERR_UNSUPPORTED, "aligned")
    expect(lib, norm_rope(lib, q=False), _lib.ERR_INVALID_ARG, "NULL")
    expect(lib, norm_rope(lib, qo=T(FAKE + 0x1000000)), _lib.ERR_INVALID_ARG, "q_out overlaps")
    expect(lib, norm_rope(lib, qo=T(FAKE + 0x3000000)), _lib.ERR_INVALID_ARG, "q_out overlaps k_out")
    expect(lib, norm_rope(lib, ko=T(FAKE + 0x6000000)), _lib.ERR_INVALID_ARG, "k_out overlaps")
    expect(lib, norm_rope(lib, qo=T(FAKE + 0x2000000, ss=0)), _lib.ERR_INVALID_ARG, "overlapping rows")
    expect(lib, norm_rope(lib, qo=T(FAKE + 0x10, S=64)), _lib.ERR_INVALID_ARG, "q_out overlaps")  # partial alias
    expect(lib, norm_rope(lib, B=0), _lib.OK)
    expect(lib, norm_rope(lib, S=0), _lib.OK)


@pytest.mark.skipif(has_gpu_node(), reason="would reach a launch on fake addresses on a GPU machine")
def test_norm_rope_in_place_passes_validation(lib):
    # exact aliasing of an output with its own input is allowed: validation
    # passes and the device query is what fails here
    expect(lib, norm_rope(lib, qo=T(FAKE), ko=T(FAKE + 0x1000000)), _lib.ERR_HIP, "hip")


def ring(lib, q=None, k=None, v=None, run=None, lse=FAKE + 0x4000000, out=False, dtype=_lib.F32, B=1, H=2, Sq=64,
         Skv=64, D=128, scale=0.088):
    q = q if q is not None else T(FAKE, S=Sq, H=H, D=D)
    k = k if k is not None else T(FAKE + 0x1000000, S=Skv, H=H, D=D)
    v = v if v is not None else T(FAKE + 0x2000000, S=Skv, H=H, D=D)
    run = run if run is not None else T(FAKE + 0x3000000, S=Sq, H=H, D=D)
    byref = lambda t: ctypes.byref(t) if t is not False else None  # noqa: E731
    return lib.regenvc_attn_ring_accumulate(byref(q), byref(k), byref(v), byref(run), lse, byref(out), dtype,
                                            B, H, Sq, Skv, D, scale, None)


def test_ring_accumulate_validation(lib):
    expect(lib, ring(lib, run=False), _lib.ERR_INVALID_ARG, "o_run")
    expect(lib, ring(lib, lse=None), _lib.ERR_INVALID_ARG, "required")
    expect(lib, ring(lib, dtype=_lib.BF16), _lib.ERR_INVALID_ARG, "F32")      # o_run is f32: no bf16 write-back
    expect(lib, ring(lib, Skv=0), _lib.ERR_INVALID_ARG, "key count")
    expect(lib, ring(lib, D=96), _lib.ERR_UNSUPPORTED, "head dim")
    expect(lib, ring(lib, run=T(FAKE + 0x3000008)), _lib.ERR_UNSUPPORTED, "aligned")
    expect(lib, ring(lib, run=T(FAKE + 0x1000000)), _lib.ERR_INVALID_ARG, "overlaps")      # o_run on k
    expect(lib, ring(lib, run=T(FAKE + 0x3000000, ss=0)), _lib.ERR_INVALID_ARG, "overlapping rows")
    expect(lib, ring(lib, lse=FAKE + 0x3000000 + 64), _lib.ERR_INVALID_ARG, "overlaps")   # lse inside o_run
    # a separate output must not overlap the running output unless it is that very view in f32
    expect(lib, ring(lib, out=T(FAKE + 0x3000000 + 256), dtype=_lib.BF16), _lib.ERR_INVALID_ARG, "o_run")
    expect(lib, ring(lib, out=T(FAKE + 0x3000000), dtype=_lib.BF16), _lib.ERR_INVALID_ARG, "o_run")
    expect(lib, ring(lib, out=T(FAKE + 0x5000000), dtype=_lib.BF16, B=0), _lib.OK)
    expect(lib, ring(lib, Sq=0), _lib.OK)


@pytest.mark.skipif(has_gpu_node(), reason="would reach a launch on fake addresses on a GPU machine")
def test_ring_accumulate_in_place_and_separate_output_pass_validation(lib):
    expect(lib, ring(lib), _lib.ERR_HIP, "hip")
    expect(lib, ring(lib, out=T(FAKE + 0x3000000), dtype=_lib.F32), _lib.ERR_HIP, "hip")
    expect(lib, ring(lib, out=T(FAKE + 0x5000000), dtype=_lib.BF16), _lib.ERR_HIP, "hip")


def dual(lib, q=None, kt=None, vt=None, ki=None, vi=None, o=None, lt=None, li=None, St=64, Si=33, B=1, H=2, Sq=64,
         D=128, scale=0.088):
    q = q if q is not None else T(FAKE, S=Sq, H=H, D=D)
    kt = kt if kt is not None else T(FAKE + 0x1000000, S=St, H=H, D=D)
    vt = vt if vt is not None else T(FAKE + 0x2000000, S=St, H=H, D=D)
    ki = ki if ki is not None else T(FAKE + 0x7000000, S=Si, H=H, D=D)
    vi = vi if vi is not None else T(FAKE + 0x8000000, S=Si, H=H, D=D)
    o = o if o is not None else T(FAKE + 0x3000000, S=Sq, H=H, D=D)
    byref = lambda t: ctypes.byref(t) if t is not False else None  # noqa: E731
    return lib.regenvc_cross_attn_dual_fwd(byref(q), byref(kt), byref(vt), St, byref(ki), byref(vi), Si, byref(o),
                                           lt, li, B, H, Sq, D, scale, None)


def test_cross_attn_dual_validation(lib):
    expect(lib, dual(lib, ki=False), _lib.ERR_INVALID_ARG, "NULL")
    expect(lib, dual(lib, Si=0), _lib.ERR_INVALID_ARG, "second context")
    expect(lib, dual(lib, St=0), _lib.ERR_INVALID_ARG, "key count")
    expect(lib, dual(lib, D=96), _lib.ERR_UNSUPPORTED, "head dim")
    expect(lib, dual(lib, vi=T(FAKE + 0x8000000, ss=100)), _lib.ERR_UNSUPPORTED, "multiple of 8")
    expect(lib, dual(lib, ki=T(FAKE + 0x7000008)), _lib.ERR_UNSUPPORTED, "aligned")
    expect(lib, dual(lib, o=T(FAKE + 0x7000000)), _lib.ERR_INVALID_ARG, "overlaps")        # o on k_img
    expect(lib, dual(lib, li=FAKE + 0x4000002), _lib.ERR_UNSUPPORTED, "aligned")
    expect(lib, dual(lib, li=FAKE + 0x8000000), _lib.ERR_INVALID_ARG, "lse_img overlaps")  # on v_img
    expect(lib, dual(lib, lt=FAKE + 0x4000000, li=FAKE + 0x4000000 + 64), _lib.ERR_INVALID_ARG, "lse_img overlaps")
    expect(lib, dual(lib, lt=FAKE + 0x7000000), _lib.ERR_INVALID_ARG, "lse overlaps")      # lse_txt on k_img
    expect(lib, dual(lib, B=0), _lib.OK)
    expect(lib, dual(lib, Sq=0, ki=False), _lib.ERR_INVALID_ARG, "NULL")


@pytest.mark.skipif(has_gpu_node(), reason="would reach a launch on fake addresses on a GPU machine")
def test_cross_attn_dual_valid_arguments_reach_the_device_check(lib):
    expect(lib, dual(lib, lt=FAKE + 0x4000000, li=FAKE + 0x4100000), _lib.ERR_HIP, "hip")


def test_workspace_binding_validation(lib):
    """regenvc_attn_set_workspace is host-only: alignment and size are checked
    on the spot; NULL unbinds."""
    expect(lib, lib.regenvc_attn_set_workspace(FAKE + 16, 4096), _lib.ERR_UNSUPPORTED, "256-byte")
    expect(lib, lib.regenvc_attn_set_workspace(FAKE, -1), _lib.ERR_INVALID_ARG, "bytes")
    expect(lib, lib.regenvc_attn_set_workspace(FAKE, 1 << 20), _lib.OK)
    # a bound workspace leaves argument validation as it was (still before any HIP call)
    expect(lib, attn(lib, D=96), _lib.ERR_UNSUPPORTED, "head dim")
    expect(lib, lib.regenvc_attn_set_workspace(None, 0), _lib.OK)
    expect(lib, lib.regenvc_attn_set_workspace(None, -5), _lib.OK)  # bytes ignored when unbinding


def test_dual_plan_query(lib):
    """The dual cross-attention plan at the window shape (10920 queries, 12
    heads, 512 + 257 context tokens): 516 query tiles, 8 + 5 key tiles, two
    whole rounds on 256 CUs and the 4 leftover tiles split over both
    contexts; workspace = ranges x 256 rows x (D + 1) floats."""
    plan = _lib.AttnPlan()
    expect(lib, lib.regenvc_cross_attn_dual_plan_query(1, 12, 10920, 512, 257, 128, 256, ctypes.byref(plan)),
           _lib.OK)
    assert plan.query_tiles == 516 and plan.key_tiles == 13
    assert plan.whole_tiles == 512 and plan.split_tiles == 4 and plan.key_ranges >= 2
    assert plan.workspace_bytes == plan.split_tiles * plan.key_ranges * 256 * 129 * 4
    expect(lib, lib.regenvc_cross_attn_dual_plan_query(1, 12, 10920, 512, 0, 128, 256, ctypes.byref(plan)),
           _lib.ERR_INVALID_ARG, "S_img")
    expect(lib, lib.regenvc_cross_attn_dual_plan_query(1, 12, 10920, 0, 257, 128, 256, ctypes.byref(plan)),
           _lib.ERR_INVALID_ARG, "key count")
    expect(lib, lib.regenvc_cross_attn_dual_plan_query(1, 12, 10920, 512, 257, 96, 256, ctypes.byref(plan)),
           _lib.ERR_UNSUPPORTED, "D=96")


def test_pool_draws_is_host_only(lib):
    assert lib.regenvc_attn_pool_draws() >= 0


def partials(lib, bounds=(0, 32, 64), parts=None, lparts=None, q=None, k=None, v=None, B=1, H=2, Sq=64, Skv=64,
             D=128, scale=0.088):
    n = len(bounds) - 1
    q = q if q is not None else T(FAKE, S=Sq, H=H, D=D)
    k = k if k is not None else T(FAKE + 0x1000000, S=Skv, H=H, D=D)
    v = v if v is not None else T(FAKE + 0x2000000, S=Skv, H=H, D=D)
    parts = parts if parts is not None else [FAKE + 0x5000000 + i * 0x1000000 for i in range(max(n, 0))]
    lparts = lparts if lparts is not None else [FAKE + 0x20000000 + i * 0x100000 for i in range(max(n, 0))]
    ba = (ctypes.c_int32 * max(len(bounds), 1))(*bounds)
    pa = (ctypes.c_void_p * max(len(parts), 1))(*parts)
    la = (ctypes.c_void_p * max(len(lparts), 1))(*lparts)
    return lib.regenvc_attn_partials_fwd(ctypes.byref(q), ctypes.byref(k), ctypes.byref(v), n, ba, pa, la, B, H, Sq,
                                         Skv, D, scale, None)


def test_chunked_partials_validation(lib):
    """regenvc_attn_partials_fwd checks its chunks and part pointers before
    any HIP call."""
    expect(lib, partials(lib, bounds=(0,)), _lib.ERR_INVALID_ARG, "num_chunks")
    expect(lib, partials(lib, bounds=tuple(range(18)), Skv=64), _lib.ERR_INVALID_ARG, "num_chunks")
    expect(lib, partials(lib, bounds=(0, 32, 32, 64)), _lib.ERR_INVALID_ARG, "empty")
    expect(lib, partials(lib, bounds=(0, 40, 20)), _lib.ERR_INVALID_ARG, "empty or reversed")
    expect(lib, partials(lib, bounds=(-1, 32, 64)), _lib.ERR_INVALID_ARG, "outside")
    expect(lib, partials(lib, bounds=(0, 32, 65)), _lib.ERR_INVALID_ARG, "outside")
    expect(lib, partials(lib, Skv=0, bounds=(0, 0, 0)), _lib.ERR_INVALID_ARG, "key count")
    expect(lib, partials(lib, parts=[FAKE + 0x5000000, 0]), _lib.ERR_INVALID_ARG, "NULL")
    expect(lib, partials(lib, parts=[FAKE + 0x5000008, FAKE + 0x6000000]), _lib.ERR_UNSUPPORTED, "aligned")
    expect(lib, partials(lib, lparts=[FAKE + 0x20000002, FAKE + 0x20100000]), _lib.ERR_UNSUPPORTED, "aligned")
    expect(lib, partials(lib, parts=[FAKE + 0x5000000, FAKE + 0x5000000 + 1024]), _lib.ERR_INVALID_ARG,
           "another part")
    expect(lib, partials(lib, parts=[FAKE + 0x1000000, FAKE + 0x6000000]), _lib.ERR_INVALID_ARG, "overlaps")
    expect(lib, partials(lib, D=96), _lib.ERR_UNSUPPORTED, "head dim")
    expect(lib, partials(lib, scale=float("nan")), _lib.ERR_INVALID_ARG, "finite")
    expect(lib, partials(lib, B=0), _lib.OK)


@pytest.mark.skipif(has_gpu_node(), reason="would reach a launch on fake addresses on a GPU machine")
def test_chunked_partials_valid_arguments_reach_the_device_check(lib):
    expect(lib, partials(lib, bounds=(3, 30, 64)), _lib.ERR_HIP, "hip")


def test_chunked_partials_plan_query(lib):
    """The rank share (H=5, 10920 queries, 4 chunks of 2730) in one launch:
    860 query tiles, 3 whole rounds on 256 CUs, the 92 leftover tiles (all in
    the last chunk) split into key ranges.  With chunks of different key tile
    counts under the split tiles, nothing is split."""
    plan = _lib.AttnPlan()
    b = (ctypes.c_int32 * 5)(0, 2730, 5460, 8190, 10920)
    expect(lib, lib.regenvc_attn_partials_plan_query(1, 5, 10920, 4, b, 128, 256, ctypes.byref(plan)), _lib.OK)
    assert plan.tile_rows == 256 and plan.query_tiles == 860 and plan.key_tiles == 43
    assert plan.whole_tiles == 768 and plan.split_tiles == 92 and plan.key_ranges >= 2
    assert plan.workspace_bytes == plan.split_tiles * plan.key_ranges * 256 * 129 * 4
    # short chunks (6 key tiles in the last): 128-row tiles, two per CU; 144 tiles on 512 slots are
    # all split candidates, and chunk 0 has 1 key tile against 6
    b = (ctypes.c_int32 * 5)(5, 69, 70, 400, 777)
    expect(lib, lib.regenvc_attn_partials_plan_query(2, 3, 700, 4, b, 128, 256, ctypes.byref(plan)), _lib.OK)
    assert plan.tile_rows == 128 and plan.query_tiles == 144 and plan.split_tiles == 0
    assert plan.workspace_bytes == 0
    # equal key tile counts: the same tiles are split
    b = (ctypes.c_int32 * 4)(0, 3000, 6000, 9000)
    expect(lib, lib.regenvc_attn_partials_plan_query(1, 2, 1000, 3, b, 128, 256, ctypes.byref(plan)), _lib.OK)
    assert plan.query_tiles == 24 and plan.split_tiles > 0 and plan.key_ranges >= 2
    # one chunk: the plain partial's plan
    b = (ctypes.c_int32 * 2)(100, 2830)
    p1 = _lib.AttnPlan()
    expect(lib, lib.regenvc_attn_partials_plan_query(1, 5, 10920, 1, b, 128, 256, ctypes.byref(plan)), _lib.OK)
    expect(lib, lib.regenvc_attn_plan_query(1, 5, 10920, 2730, 128, 256, ctypes.byref(p1)), _lib.OK)
    assert {f: getattr(plan, f) for f, _ in plan._fields_} == {f: getattr(p1, f) for f, _ in p1._fields_}
    b = (ctypes.c_int32 * 3)(0, 10, 10)
    expect(lib, lib.regenvc_attn_partials_plan_query(1, 5, 10920, 2, b, 128, 256, ctypes.byref(plan)),
           _lib.ERR_INVALID_ARG, "empty")
