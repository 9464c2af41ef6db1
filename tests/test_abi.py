"""The C ABI on the CPU: exports, validation and status codes, with no GPU work.

Every check in ``stencil_plan``/``stencil_apply`` happens on the host before the first HIP
call, so invalid calls are tested here with placeholder device addresses that the library
never dereferences.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2608_21157_amd import binding as B

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                      "stencil.h")

IN, OUT, FIELD = 0x7F0000000000, 0x7F0100000000, 0x7F0200000000  # never dereferenced


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(stencil_\w+)\s*\(", text)))


def desc3(**kw):
    base = dict(batch=1, channels=1, dtype=B.F32, shape=B.STAR, radius=1, boundary=B.ZERO)
    base.update(kw)
    dims = base.pop("dims", (8, 8, 8))
    return B.make_desc(3, dims, **base)


def status_of(fn, *args):
    try:
        fn(*args)
    except B.StencilError as e:
        return e.status
    return B.OK


def test_library_exports_every_declared_function():
    lib = B.load()
    declared = header_functions()
    assert set(declared) == set(B.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name


def test_status_strings_and_point_counts():
    assert B.stencil_status_str(B.OK) == "STENCIL_OK"
    assert B.stencil_status_str(B.ERR_ALIAS) == "STENCIL_ERR_ALIAS"
    assert B.stencil_status_str(99) == "unknown status"
    assert B.stencil_num_points(B.STAR, 3, 4) == 25
    assert B.stencil_num_points(B.BOX, 3, 1) == 27
    assert B.stencil_num_points(B.BOX, 2, 3) == 49
    assert B.stencil_num_points(B.STAR, 2, 1) == 5
    assert B.stencil_num_points(B.STAR, 4, 1) == -1


@pytest.mark.parametrize("kw,status", [
    (dict(dims=(0, 8, 8)), B.ERR_INVALID_ARG),
    (dict(batch=0), B.ERR_INVALID_ARG),
    (dict(channels=0), B.ERR_INVALID_ARG),
    (dict(dtype=2), B.ERR_INVALID_ARG),
    (dict(shape=5), B.ERR_INVALID_ARG),
    (dict(boundary=3), B.ERR_INVALID_ARG),
    (dict(radius=-1), B.ERR_INVALID_ARG),
    (dict(radius=5), B.ERR_UNSUPPORTED),
    (dict(shape=B.BOX, radius=4), B.ERR_UNSUPPORTED),
    (dict(variant=7), B.ERR_INVALID_ARG),
    (dict(temporal_depth=-1), B.ERR_INVALID_ARG),
    (dict(variant=B.VARIANT_GENERIC, temporal_depth=2), B.ERR_UNSUPPORTED),
    (dict(shape=B.STAR, radius=1, temporal_depth=5), B.ERR_UNSUPPORTED),    # at most 4
    (dict(shape=B.STAR, radius=2, temporal_depth=3), B.ERR_UNSUPPORTED),    # radius 1 only
    (dict(shape=B.STAR, radius=1, dtype=B.F64, temporal_depth=4), B.ERR_UNSUPPORTED),
    (dict(dims=(1 << 11, 1 << 11, 1 << 11)), B.ERR_UNSUPPORTED),
    (dict(tile=3), B.ERR_INVALID_ARG),
    (dict(tile=-1), B.ERR_INVALID_ARG),
    (dict(grid_scale=3), B.ERR_INVALID_ARG),
    (dict(grid_scale=-3), B.ERR_INVALID_ARG),
    (dict(variant=B.VARIANT_GENERIC, tile=1), B.ERR_UNSUPPORTED),
    (dict(dims=(8, 8, 10), tile=2), B.ERR_UNSUPPORTED),          # generic only (x % 4)
])
def test_plan_rejects(kw, status):
    assert status_of(B.stencil_plan, desc3(**kw)) == status
    assert B.stencil_status_str(status) in B.stencil_last_error()


def test_plan_rejects_bad_ndim_and_null():
    d = desc3()
    d.ndim = 4
    assert status_of(B.stencil_plan, d) == B.ERR_INVALID_ARG
    h = ctypes.c_void_p(123)
    assert B.load().stencil_plan(None, ctypes.byref(h)) == B.ERR_INVALID_ARG
    assert h.value is None
    assert B.load().stencil_plan(ctypes.byref(desc3()), None) == B.ERR_INVALID_ARG


def test_forced_stream_variant_rejects_what_it_cannot_tile():
    for d in (B.make_desc(2, (64, 66), shape=B.BOX, radius=3, variant=B.VARIANT_STREAM),  # x % 4
              B.make_desc(2, (64, 4 * 96), shape=B.BOX, radius=3, variant=B.VARIANT_STREAM),
              B.make_desc(2, (64, 64), shape=B.BOX, radius=3, has_coeff_field=True,
                          variant=B.VARIANT_STREAM),
              B.make_desc(3, (8, 8, 10), shape=B.STAR, variant=B.VARIANT_STREAM),  # x % 4
              B.make_desc(3, (8, 8, 8), shape=B.BOX, radius=2, variant=B.VARIANT_STREAM)):
        assert status_of(B.stencil_plan, d) == B.ERR_UNSUPPORTED


def test_planner_choices():
    """The planner picks the tiled kernel family and temporal depth per description."""
    cases = [
        (B.make_desc(3, (512,) * 3, shape=B.STAR, radius=4), "stencil_star_tb2_kernel", 2),
        (B.make_desc(3, (512,) * 3, shape=B.STAR, radius=4, temporal_depth=1),
         "stencil_star_stream_kernel", 1),
        (B.make_desc(3, (256,) * 3, shape=B.STAR, radius=1), "stencil_star_tb2_kernel", 2),
        (B.make_desc(3, (512,) * 3, shape=B.BOX, radius=1, has_coeff_field=True,
                     boundary=B.PERIODIC), "stencil_box3_stream_kernel", 1),
        (B.make_desc(3, (128,) * 3, batch=256, channels=32, shape=B.BOX, radius=1),
         "stencil_box3_stream_kernel", 1),
        (B.make_desc(2, (10240, 10240), shape=B.BOX, radius=3, dtype=B.F64),
         "stencil_box2_tb2_kernel", 2),
        (B.make_desc(2, (10240, 10240), shape=B.BOX, radius=3, dtype=B.F64, temporal_depth=1),
         "stencil_box2_stream_kernel", 1),
        (B.make_desc(2, (256, 256), shape=B.STAR, radius=1), "stencil_star_stream_kernel", 1),
        (B.make_desc(3, (8, 8, 10), shape=B.STAR, radius=1), "stencil_generic_kernel", 1),
        (B.make_desc(3, (256,) * 3, shape=B.STAR, radius=4, temporal_depth=2),
         "stencil_star_tb2_kernel", 2),
        # fp32 radius 1 beyond the Infinity Cache: four steps per pass; inside it, two
        (B.make_desc(3, (512,) * 3, shape=B.STAR, radius=1), "stencil_star_tbs_kernel", 4),
        (B.make_desc(3, (256,) * 3, shape=B.STAR, radius=1, temporal_depth=4),
         "stencil_star_tbs_kernel", 4),
        (B.make_desc(3, (256,) * 3, shape=B.STAR, radius=1, temporal_depth=3),
         "stencil_star_tbs_kernel", 3),
        (B.make_desc(3, (512,) * 3, shape=B.STAR, radius=1, dtype=B.F64),
         "stencil_star_tbs_kernel", 3),
        (B.make_desc(3, (64, 256, 256), shape=B.STAR, radius=1, dtype=B.F64),
         "stencil_star_tb2_kernel", 2),
        (B.make_desc(3, (512,) * 3, shape=B.STAR, radius=2), "stencil_star_tb2_kernel", 2),
    ]
    for d, kernel, depth in cases:
        h = B.stencil_plan(d)
        info = B.stencil_plan_query(h)
        assert info.kernel.decode() == kernel and info.temporal_depth == depth
        B.stencil_destroy(h)


def test_plan_and_query_without_gpu():
    h = B.stencil_plan(B.make_desc(2, (16, 18), shape=B.BOX, radius=3, dtype=B.F64))
    info = B.stencil_plan_query(h)
    assert info.variant == B.VARIANT_GENERIC and info.temporal_depth == 1
    assert info.scratch_bytes == 16 * 18 * 8
    assert info.kernel.decode() == "stencil_generic_kernel"
    B.stencil_destroy(h)
    B.stencil_destroy(None)


def test_tile_and_grid_scale_choices():
    """tile is accepted where the one-step kernel has two (3D star, 3D box), refused for the
    2D box family; grid_scale is accepted by every variant; the plan reports both."""
    for d, tile in ((desc3(dims=(64, 64, 256), radius=4, tile=1, grid_scale=-2), 1),
                    (desc3(dims=(64, 64, 256), shape=B.BOX, tile=2, grid_scale=2), 2),
                    (desc3(dims=(8, 8, 10), grid_scale=1), 0),
                    # 0 resolved: 8 rows per lane for the box (4 with a field), 64 x 64
                    # tiles for the one-step 3D star, 64 x 32 in 2D; the fused star has
                    # one tile
                    (desc3(dims=(64, 64, 256), shape=B.BOX), 2),
                    (desc3(dims=(64, 64, 256), shape=B.BOX, has_coeff_field=True), 1),
                    (desc3(dims=(64, 64, 256), radius=4, temporal_depth=1), 2),
                    (B.make_desc(2, (256, 256), radius=1), 1),
                    (desc3(dims=(64, 64, 256), radius=4), 0)):
        h = B.stencil_plan(d)
        info = B.stencil_plan_query(h)
        assert (info.tile, info.grid_scale) == (tile, d.grid_scale)
        B.stencil_destroy(h)
    box2 = B.make_desc(2, (1024, 1024), shape=B.BOX, radius=3, dtype=B.F64, tile=1)
    assert status_of(B.stencil_plan, box2) == B.ERR_UNSUPPORTED
    assert "single tile" in B.stencil_last_error()


@pytest.fixture
def plan():
    h = B.stencil_plan(desc3(dims=(4, 5, 6), shape=B.BOX, radius=1, has_coeff_field=True))
    yield h
    B.stencil_destroy(h)


W27 = np.zeros(27, np.float32)


def apply_status(h, inp=IN, out=OUT, dims=(4, 5, 6), coeffs=W27, field=FIELD, radius=1,
                 boundary=B.ZERO, steps=1):
    return status_of(B.stencil_apply, h, inp, out, dims, coeffs, field, radius, boundary, steps,
                     None)


def test_apply_validation(plan):
    assert apply_status(None) == B.ERR_INVALID_ARG
    assert apply_status(plan, inp=None) == B.ERR_INVALID_ARG
    assert apply_status(plan, out=None) == B.ERR_INVALID_ARG
    assert apply_status(plan, coeffs=None) == B.ERR_INVALID_ARG
    assert apply_status(plan, steps=-1) == B.ERR_INVALID_ARG
    assert apply_status(plan, dims=(4, 5, 7)) == B.ERR_MISMATCH
    assert apply_status(plan, radius=2) == B.ERR_MISMATCH
    assert apply_status(plan, boundary=B.PERIODIC) == B.ERR_MISMATCH
    assert apply_status(plan, field=None) == B.ERR_MISMATCH
    assert apply_status(plan, out=IN) == B.ERR_ALIAS
    assert apply_status(plan, out=IN + 4 * 100) == B.ERR_ALIAS         # partial overlap
    assert apply_status(plan, out=IN + 4 * 120) != B.ERR_ALIAS         # just past the end
    assert apply_status(plan, out=FIELD + 8) == B.ERR_ALIAS
    assert "overlaps" in B.stencil_last_error()
    d = (ctypes.c_int64 * 3)(4, 5, 6)
    assert B.load().stencil_apply(plan, IN, OUT, None, W27.ctypes.data, FIELD, 1, 0, 1,
                                  None) == B.ERR_INVALID_ARG
    assert B.load().stencil_apply(plan, IN, OUT, d, W27.ctypes.data, None, 1, 0, 1,
                                  None) == B.ERR_MISMATCH


def test_field_given_to_plan_without_field():
    h = B.stencil_plan(desc3(dims=(4, 5, 6)))
    try:
        assert apply_status(h, coeffs=np.zeros(7, np.float32)) == B.ERR_MISMATCH
    finally:
        B.stencil_destroy(h)


def test_valid_apply_without_gpu_reports_hip_error(plan):
    """All checks pass, then the first HIP call fails cleanly on a host with no GPU."""
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    assert apply_status(plan) == B.ERR_HIP
    assert "hipGetDevice" in B.stencil_last_error()


def tune_status(h, inp=IN, out=OUT, dims=(4, 5, 6), coeffs=W27, field=FIELD, steps=1,
                tolerance=-1.0, reps=0, report=None):
    return status_of(B.stencil_tune, h, inp, out, dims, coeffs, field, steps, tolerance, reps,
                     None, report)


def test_tune_validation(plan):
    """stencil_tune checks everything stencil_apply checks, plus its own arguments, on the
    host; a failed call leaves the report untouched and the plan unchanged."""
    rep = B.StencilTuneReport()
    rep.count = 77
    assert tune_status(None) == B.ERR_INVALID_ARG
    assert tune_status(plan, inp=None, report=rep) == B.ERR_INVALID_ARG
    assert tune_status(plan, coeffs=None) == B.ERR_INVALID_ARG
    assert tune_status(plan, dims=(4, 5, 7)) == B.ERR_MISMATCH
    assert tune_status(plan, field=None) == B.ERR_MISMATCH
    assert tune_status(plan, out=IN + 8) == B.ERR_ALIAS
    assert tune_status(plan, steps=0) == B.ERR_INVALID_ARG
    assert "steps >= 1" in B.stencil_last_error()
    assert tune_status(plan, reps=-1) == B.ERR_INVALID_ARG
    assert tune_status(plan, reps=1001) == B.ERR_INVALID_ARG
    assert tune_status(plan, tolerance=float("nan")) == B.ERR_INVALID_ARG
    assert rep.count == 77
    info = B.stencil_plan_query(plan)
    assert (info.variant, info.temporal_depth, info.tile, info.grid_scale) == (
        B.VARIANT_STREAM, 1, 0, 0) or info.variant == B.VARIANT_GENERIC


def test_valid_tune_without_gpu_reports_hip_error(plan):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    assert tune_status(plan, steps=2) == B.ERR_HIP
    assert "hipGetDevice" in B.stencil_last_error()


def noalloc_status(h, inp=IN, out=OUT, dims=(4, 5, 6), coeffs=W27, field=FIELD, radius=1,
                   boundary=B.ZERO, steps=1):
    return status_of(B.stencil_apply_noalloc, h, inp, out, dims, coeffs, field, radius,
                     boundary, steps, None)


def test_noalloc_validation_matches_apply(plan):
    """The allocation-free entry point makes stencil_apply's checks, with its statuses."""
    for kw in (dict(inp=None), dict(coeffs=None), dict(steps=-1), dict(dims=(4, 5, 7)),
               dict(radius=2), dict(boundary=B.PERIODIC), dict(field=None), dict(out=IN),
               dict(out=FIELD + 8)):
        assert noalloc_status(plan, **kw) == apply_status(plan, **kw) != B.OK
    assert noalloc_status(None) == B.ERR_INVALID_ARG


def test_noalloc_scratch_limits_are_checked_before_any_hip_call():
    """A call that needs an intermediate grid larger than the static scratch, or weights
    larger than its weight region, is refused on the host, even without a GPU."""
    limit = B.NOALLOC_GRID_BYTES
    # 256^3 fp32 is exactly the grid region: its multi-launch calls fit
    fits = B.stencil_plan(desc3(dims=(256, 256, 256)))
    big = B.stencil_plan(desc3(dims=(257, 256, 256)))
    w7 = np.zeros(7, np.float32)
    try:
        assert 256 ** 3 * 4 == limit
        # beyond the Infinity Cache the planner fuses four steps per launch
        assert B.stencil_plan_query(big).temporal_depth == 4
        kw = dict(dims=(257, 256, 256), coeffs=w7, field=None, out=OUT + (1 << 30))
        assert noalloc_status(big, steps=5, **kw) == B.ERR_UNSUPPORTED   # 2 launches
        assert "intermediate grid" in B.stencil_last_error()
        import torch
        if not torch.cuda.is_available():
            # one launch (four fused steps) and 0 steps need no grid: they reach HIP
            assert noalloc_status(big, steps=4, **kw) == B.ERR_HIP
            assert noalloc_status(big, steps=0, **kw) == B.ERR_HIP
            kw["dims"] = (256, 256, 256)
            assert noalloc_status(fits, steps=5, **kw) == B.ERR_HIP
    finally:
        B.stencil_destroy(fits)
        B.stencil_destroy(big)
    # 64 KiB of weights: 304 weight sets of 27 fp64 values do not fit, 303 do
    for channels, status in ((304, B.ERR_UNSUPPORTED), (303, B.ERR_HIP)):
        h = B.stencil_plan(desc3(dims=(4, 5, 6), shape=B.BOX, dtype=B.F64, batch=channels,
                                 channels=channels))
        try:
            import torch
            if status == B.ERR_HIP and torch.cuda.is_available():
                continue
            w = np.zeros(channels * 27, np.float64)
            assert noalloc_status(h, coeffs=w, field=None, out=OUT + (1 << 30)) == status
        finally:
            B.stencil_destroy(h)
    assert 303 * 27 * 8 <= B.NOALLOC_WEIGHT_BYTES < 304 * 27 * 8


def test_noalloc_limits_match_the_header():
    text = open(HEADER).read()
    assert re.search(r"STENCIL_NOALLOC_WEIGHT_BYTES \(64 \* 1024\)", text)
    assert re.search(r"STENCIL_NOALLOC_GRID_BYTES \(64 \* 1024 \* 1024\)", text)
    assert B.NOALLOC_WEIGHT_BYTES == 64 * 1024 and B.NOALLOC_GRID_BYTES == 64 << 20
