"""Shared helpers of the GPU parity tests: run the library through the C ABI, pick sample
points, and state the tolerance.

Tolerance (fp32): max |gpu - oracle| <= 1e-5 * max(steps, 1) * max(1, max|x|) * max(1, max k).
The 1e-5-per-step bar assumes inputs in [-1, 1] and sum|w| <= 1; inputs of larger magnitude
(the N(0,1) conv-form workload) scale it by max|x|.  The worst-case fp32 rounding of a
27-term sum is 27 * 2^-24 * sum|w| * max|x| ~ 1.6e-6 * max|x|, below the bar.
Tolerance (fp64): 1e-12 * max(steps, 1) * max(1, max|x|).
"""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2608_21157_amd import binding as B


def tolerance(wl, x, k=None, steps=None) -> float:
    steps = wl.steps if steps is None else steps
    scale = max(1.0, float(np.abs(x).max()) if x.size else 1.0)
    if k is not None:
        scale *= max(1.0, float(np.abs(k).max()))
    base = 1e-5 if wl.dtype == "f32" else 1e-12
    return base * max(steps, 1) * scale


def run_library(wl, x, w, k=None, *, steps=None, variant=B.VARIANT_AUTO, depth=0,
                stream=None, tile=0, grid_scale=0):
    """Upload, apply through the C ABI, download.  Returns (result float64, plan info)."""
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
    return yt.cpu().numpy().astype(np.float64), info


def oracle_full(wl, x, w, k=None, steps=None):
    steps = wl.steps if steps is None else steps
    return oracle.apply(x, w, shape=wl.shape, radius=wl.radius, boundary=wl.boundary,
                        steps=steps, field=k, ndim=wl.ndim, channels=wl.channels)


def sample_points(wl, x, count: int, seed: int = 0, steps=None):
    """Sample (b, z, y, x) rows: all corners, points within R*steps of each face, and
    uniformly random interior points."""
    steps = wl.steps if steps is None else steps
    g = np.random.default_rng(seed)
    dims = (1,) + tuple(wl.dims) if wl.ndim == 2 else tuple(wl.dims)
    lead = x.shape[: x.ndim - wl.ndim]
    batch = int(np.prod(lead)) if len(lead) else 1
    reach = wl.radius * max(steps, 1) + 1
    pts = []
    for b in sorted({0, batch - 1}):
        for cz in sorted({0, dims[0] - 1}):
            for cy in (0, dims[1] - 1):
                for cx in (0, dims[2] - 1):
                    pts.append((b, cz, cy, cx))
    for _ in range(count // 2):   # near a face along one random axis
        p = [int(g.integers(0, batch))] + [int(g.integers(0, n)) for n in dims]
        a = int(g.integers(1 if wl.ndim == 3 else 2, 4))
        d = int(g.integers(0, min(reach, dims[a - 1])))
        p[a] = d if g.random() < 0.5 else dims[a - 1] - 1 - d
        pts.append(tuple(p))
    for _ in range(count - count // 2):
        pts.append((int(g.integers(0, batch)),) + tuple(int(g.integers(0, n)) for n in dims))
    return np.array(pts, dtype=np.int64)


def gather(result, pts, wl):
    """Values of a (batch?, *dims) result at (b, z, y, x) rows."""
    dims = tuple(wl.dims)
    flat = result.reshape((-1,) + dims)
    if wl.ndim == 2:
        return flat[pts[:, 0], pts[:, 2], pts[:, 3]]
    return flat[pts[:, 0], pts[:, 1], pts[:, 2], pts[:, 3]]


def report(name, got, ref, tol):
    err = np.abs(got - ref)
    i = int(np.nanargmax(err)) if err.size else 0
    worst = float(err.flat[i]) if err.size else 0.0
    rel = worst / max(abs(float(ref.flat[i])), 1e-30) if err.size else 0.0
    print("[parity] %s max_abs_err=%.3e (rel %.2e at flat %d) tol=%.1e" % (name, worst, rel, i,
                                                                          tol), flush=True)
    assert np.isfinite(got).all(), "%s: non-finite values" % name
    assert worst <= tol, "%s: max abs error %.3e > %.1e" % (name, worst, tol)
