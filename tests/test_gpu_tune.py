"""The plan-time tuner (stencil_tune) and the launch knobs it searches (tile, grid_scale),
on the GPU, against the oracle.

The tuner mirrors the validity-gated search of HIERA (Sec. "Problem Formulation and
Framework Overview", Eq. 2): among the explored candidates, the fastest one whose result
stays within tolerance of the reference.  These tests check that the gate and the choice
do what stencil.h says, and that every launch configuration the tuner can pick computes
the operator (oracle parity), so a tuned plan is as correct as an untuned one.
"""
import numpy as np
import pytest
import torch

from paper_2608_21157_amd import binding as B
from paper_2608_21157_amd import inputs
from paper_2608_21157_amd.inputs import WORKLOADS
from parity_util import oracle_full, report, run_library, tolerance

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def case(name, dims, steps=None, n=None):
    wl = WORKLOADS[name].resized(dims, n=n, steps=steps)
    return wl, inputs.make(wl)


def desc_of(wl, x, k, **kw):
    lead = x.shape[: x.ndim - wl.ndim]
    batch = int(np.prod(lead)) if len(lead) else 1
    return B.make_desc(wl.ndim, wl.dims, batch=batch, channels=wl.channels,
                       dtype=B.F32 if wl.dtype == "f32" else B.F64, shape=wl.shape,
                       radius=wl.radius, boundary=wl.boundary, has_coeff_field=k is not None,
                       **kw)


def tune(wl, x, w, k, *, tolerance_=-1.0, reps=2, offset=0):
    """Tune a fresh plan on device copies of x (and k); `offset` elements of misalignment.
    Returns (report, plan info, tuned output, output of a later run of the tuned plan)."""
    n = x.size
    base = torch.empty(n + offset, dtype=torch.float32 if wl.dtype == "f32" else torch.float64,
                       device=DEV)
    xt = base[offset:].view(x.shape)
    xt.copy_(torch.from_numpy(np.ascontiguousarray(x)))
    ybase = torch.full_like(base, float("nan"))
    yt = ybase[offset:].view(x.shape)
    kt = None if k is None else torch.from_numpy(np.ascontiguousarray(k)).to(DEV)
    plan = B.Plan(desc_of(wl, x, k))
    try:
        rep = plan.tune(xt, yt, w, steps=wl.steps, field=kt, tolerance=tolerance_, reps=reps)
        info = plan.info()
        y2 = torch.full_like(yt, float("nan"))
        plan.run(xt, y2, w, steps=wl.steps, field=kt)
        torch.cuda.synchronize()
    finally:
        plan.close()
    print("[tune] %s tol=%.2e chosen=%d" % (wl.name, rep["tolerance"], rep["chosen"]), flush=True)
    for i, c in enumerate(rep["candidates"]):
        print("[tune]   %2d %s" % (i, c), flush=True)
    return rep, info, yt.cpu().numpy().astype(np.float64), y2.cpu().numpy().astype(np.float64)


TUNE_CASES = [
    # name, dims, steps, candidates: generic + depth 1 (tiles x 4 scales) + depth 2 (4 scales)
    # (+ depth 4, 4 scales, for fp32 radius-1 stars)
    ("c3", (40, 48, 256), 3, 1 + 2 * 4 + 4),
    ("c2", (24, 40, 64), 5, 1 + 2 * 4 + 4 + 4),
    ("c4", (12, 20, 512), None, 1 + 2 * 4),
    ("paper", (96, 512), 3, 1 + 4 + 4),
]


@pytest.mark.parametrize("name,dims,steps,count", TUNE_CASES, ids=[c[0] for c in TUNE_CASES])
def test_tune_fixes_fastest_valid_candidate(name, dims, steps, count):
    wl, (x, w, k) = case(name, dims, steps)
    rep, info, y, y2 = tune(wl, x, w, k)
    cands = rep["candidates"]
    assert len(cands) == count
    assert cands[0]["variant"] == "generic" and cands[0]["max_abs_err"] == 0.0
    assert all(c["valid"] and c["ms"] > 0 for c in cands), "a kernel failed the default gate"
    assert all(c["max_abs_err"] <= rep["tolerance"] for c in cands)
    chosen = cands[rep["chosen"]]
    assert chosen["ms"] == min(c["ms"] for c in cands)
    assert (B.VARIANT_NAMES[info.variant], info.temporal_depth, info.tile, info.grid_scale) == (
        chosen["variant"], chosen["temporal_depth"], chosen["tile"], chosen["grid_scale"])
    ref = oracle_full(wl, x, w, k)
    tol = tolerance(wl, x, k)
    report("%s tuned output" % name, y, ref, tol)
    report("%s tuned plan, second run" % name, y2, ref, tol)


def test_tune_gate_rejects_candidates_beyond_the_tolerance():
    """With an explicit tolerance below some candidates' error, exactly those candidates
    fail the gate and are not timed; tolerance 0 keeps only results identical to the
    reference (the reference itself always passes)."""
    wl, (x, w, k) = case("c3", (40, 48, 256), 3)
    first, _, _, _ = tune(wl, x, w, k)
    errs = sorted({c["max_abs_err"] for c in first["candidates"] if c["max_abs_err"] > 0})
    for tol in ([0.0] + ([errs[0] / 2] if errs else [])):
        rep, info, y, _ = tune(wl, x, w, k, tolerance_=tol)
        assert rep["tolerance"] == tol
        for c in rep["candidates"]:
            assert c["valid"] == (c["max_abs_err"] <= tol)
            assert (c["ms"] > 0) == c["valid"]
        assert rep["candidates"][0]["valid"]
        assert rep["candidates"][rep["chosen"]]["max_abs_err"] <= tol
        report("tolerance %.1e output" % tol, y, oracle_full(wl, x, w, k), tolerance(wl, x, k))
    if not errs:
        pytest.skip("every kernel matched the reference bit for bit; nothing to reject")
    assert any(not c["valid"] for c in rep["candidates"])


def test_tune_misaligned_buffers_offer_only_the_generic_kernel():
    wl, (x, w, k) = case("c3", (16, 16, 64), 2)
    rep, info, y, _ = tune(wl, x, w, k, offset=1)
    assert len(rep["candidates"]) == 1 and rep["chosen"] == 0
    assert info.variant == B.VARIANT_GENERIC
    report("misaligned tune", y, oracle_full(wl, x, w, k), tolerance(wl, x, k))


def test_tune_leaves_plan_unchanged_when_nothing_passes():
    """An input with a NaN makes every candidate's error NaN, which never passes the gate:
    the call reports UNSUPPORTED and the plan keeps its choice."""
    wl, (x, w, k) = case("c3", (16, 16, 64), 2)
    x = x.copy()
    x[3, 4, 5] = np.nan
    xt = torch.from_numpy(x).to(DEV)
    yt = torch.empty_like(xt)
    plan = B.Plan(desc_of(wl, x, None))
    before = plan.info()
    try:
        with pytest.raises(B.StencilError) as ei:
            plan.tune(xt, yt, w, steps=wl.steps, tolerance=1.0)
        assert ei.value.status == B.ERR_UNSUPPORTED
        after = plan.info()
        assert (after.variant, after.temporal_depth, after.tile, after.grid_scale) == (
            before.variant, before.temporal_depth, before.tile, before.grid_scale)
    finally:
        plan.close()


KNOB_CASES = [
    # name, dims, steps, depth, tile, grid_scale
    ("c3", (40, 48, 256), 3, 1, 1, -2),
    ("c3", (40, 48, 256), 3, 1, 2, 2),
    ("c3", (40, 48, 256), 3, 2, 0, -2),
    ("c3", (40, 48, 256), 3, 2, 0, 2),
    ("c1", (96, 256), 2, 1, 2, 1),
    ("c4", (12, 20, 512), None, 1, 1, 2),
    ("c4", (12, 20, 512), None, 1, 2, -2),
    ("c5", (16, 16, 128), None, 1, 1, -1),
    ("c5", (16, 16, 128), None, 1, 2, 2),
    ("paper", (96, 512), 3, 1, 0, -2),
    ("paper", (96, 512), 3, 2, 0, 2),
]


@pytest.mark.parametrize("name,dims,steps,depth,tile,scale", KNOB_CASES,
                         ids=["%s-d%d-t%d-s%d" % (c[0], c[3], c[4], c[5]) for c in KNOB_CASES])
def test_tile_and_grid_scale_parity(name, dims, steps, depth, tile, scale):
    """Every tile and grid scale the tuner can choose computes the operator."""
    n = 1 if name == "c5" else None
    wl, (x, w, k) = case(name, dims, steps, n=n)
    got, info = run_library(wl, x, w, k, depth=depth, tile=tile, grid_scale=scale)
    assert (info["tile"], info["grid_scale"]) == (tile, scale)
    report("%s %s" % (name, info), got, oracle_full(wl, x, w, k), tolerance(wl, x, k))


@pytest.mark.parametrize("scale", [-2, 2])
def test_generic_grid_scale_parity(scale):
    wl, (x, w, k) = case("c4", (9, 10, 44), None)
    got, info = run_library(wl, x, w, k, variant=B.VARIANT_GENERIC, grid_scale=scale)
    report("generic scale %d" % scale, got, oracle_full(wl, x, w, k), tolerance(wl, x, k))
