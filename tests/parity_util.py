"""Shared helpers of the GPU parity tests: run the library through the C ABI, compare
with the oracle (whole grids, or full-size grids piece by piece), and state the
tolerance.

Tolerance (fp32): max |gpu - oracle| <= 1e-5 * max(steps, 1) * max(1, max|x|) * max(1, max k).
The 1e-5-per-step bar assumes inputs in [-1, 1] and sum|w| <= 1; inputs of larger magnitude
(the N(0,1) conv-form workload) scale it by max|x|.  The worst-case fp32 rounding of a
27-term sum is 27 * 2^-24 * sum|w| * max|x| ~ 1.6e-6 * max|x|, below the bar.
Tolerance (fp64): a flat 1e-12, whatever the step count or the input's magnitude.  The
worst-case fp64 rounding of the largest case here (27 terms, N(0,1) input with max|x| ~ 5.4)
is 27 * 2^-53 * 5.4 ~ 1.6e-14 per step, and every multi-step workload is non-expansive
(sum|w| <= 1), so the flat bar holds with two orders of magnitude to spare.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2608_21157_amd import binding as B


FP32_PER_STEP = 1e-5
FP64_FLAT = 1e-12


def tolerance(wl, x, k=None, steps=None) -> float:
    if wl.dtype != "f32":
        return FP64_FLAT
    steps = wl.steps if steps is None else steps
    scale = max(1.0, float(np.abs(x).max()) if x.size else 1.0)
    if k is not None:
        scale *= max(1.0, float(np.abs(k).max()))
    return FP32_PER_STEP * max(steps, 1) * scale


def run_library(wl, x, w, k=None, *, steps=None, variant=B.VARIANT_AUTO, depth=0,
                stream=None, tile=0, grid_scale=0, as_f64=True):
    """Upload, apply through the C ABI, download.  Returns (result, plan info); the
    result is float64, or the computed dtype with ``as_f64=False`` (full-size grids)."""
    steps = wl.steps if steps is None else steps
    dev = torch.device("cuda:0")
    xt = torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    yt = torch.full_like(xt, float("nan"))
    kt = None if k is None else torch.from_numpy(np.ascontiguousarray(k)).to(dev)
    torch.cuda.synchronize()  # the NaN fill runs on torch's stream; the call may use another
    lead = xt.shape[: xt.dim() - wl.ndim]
    batch = int(np.prod(lead)) if len(lead) else 1
    desc = B.make_desc(wl.ndim, xt.shape[xt.dim() - wl.ndim:], batch=batch,
                       channels=wl.channels, dtype=B.F32 if wl.dtype == "f32" else B.F64,
                       shape=wl.shape, radius=wl.radius, boundary=wl.boundary,
                       has_coeff_field=k is not None, variant=variant, temporal_depth=depth,
                       tile=tile, grid_scale=grid_scale)
    plan = B.Plan(desc)
    try:
        info = plan.info()
        info = dict(variant=info.variant, depth=info.temporal_depth,
                    kernel=info.kernel.decode(), tile=info.tile, grid_scale=info.grid_scale)
        plan.run(xt, yt, w, steps=steps, field=kt, stream=stream)
        torch.cuda.synchronize()
    finally:
        plan.close()
    got = yt.cpu().numpy()
    return (got.astype(np.float64) if as_f64 else got), info


def oracle_full(wl, x, w, k=None, steps=None):
    steps = wl.steps if steps is None else steps
    return oracle.apply(x, w, shape=wl.shape, radius=wl.radius, boundary=wl.boundary,
                        steps=steps, field=k, ndim=wl.ndim, channels=wl.channels)


def dense_report(name, wl, x, w, k, got, tol, steps=None):
    """``got`` against the oracle at every point of a full-size grid: the oracle runs in
    independent slabs or volumes on host threads (``oracle/whole_grid.py``)."""
    from oracle import whole_grid
    steps = wl.steps if steps is None else steps
    rep = whole_grid.compare(got, x, w, shape=wl.shape, radius=wl.radius,
                             boundary=wl.boundary, steps=steps, ndim=wl.ndim,
                             channels=wl.channels, field=k)
    print("[parity] %s every point: %d points, max_abs_err=%.3e at flat %d, tol=%.1e, "
          "nonfinite=%d (oracle %.1f s on %d threads, %d pieces)" % (
              name, rep["points"], rep["max_abs_err"], rep["worst"], tol, rep["nonfinite"],
              rep["seconds"], rep["threads"], rep["pieces"]), flush=True)
    assert rep["points"] == x.size
    assert rep["nonfinite"] == 0, "%s: non-finite values" % name
    assert rep["max_abs_err"] <= tol, "%s: max abs error %.3e > %.1e" % (
        name, rep["max_abs_err"], tol)
    return rep


def report(name, got, ref, tol):
    err = np.abs(got - ref)
    i = int(np.nanargmax(err)) if err.size else 0
    worst = float(err.flat[i]) if err.size else 0.0
    rel = worst / max(abs(float(ref.flat[i])), 1e-30) if err.size else 0.0
    print("[parity] %s max_abs_err=%.3e (rel %.2e at flat %d) tol=%.1e" % (name, worst, rel, i,
                                                                          tol), flush=True)
    assert np.isfinite(got).all(), "%s: non-finite values" % name
    assert worst <= tol, "%s: max abs error %.3e > %.1e" % (name, worst, tol)
