"""Seeded random descriptions through the planner, every point against the oracle.

Each case draws a description: 2D or 3D, star or box, every supported radius (0 included),
fp32 or fp64, zero or periodic, a coefficient field or not, 1-3 volumes with 1-2 weight
sets, 0-5 steps, and extents from 1 to 40 rows and planes with x extents that the
streaming kernels tile (a multiple of 16 bytes, or whole 64-lane row segments) or do not.
The planner picks the kernel family and the temporal depth as it would for a caller, so
the cases cross the families' boundaries (generic fallback, one-step and fused kernels,
odd trailing steps).  The draws are fixed by the case seed; each case prints its
description before it runs.
"""
import numpy as np
import pytest

from dataclasses import replace

from paper_2608_21157_amd import binding as B
from paper_2608_21157_amd.inputs import WORKLOADS
from parity_util import oracle_full, report, run_library, tolerance

pytestmark = pytest.mark.gpu

SEEDS = list(range(120))


def draw(seed):
    g = np.random.default_rng(1000 + seed)
    # the operator family first, weighted toward those a streaming kernel runs
    fam = str(g.choice(["star3", "star2", "box3", "box2", "any"], p=[.3, .15, .2, .15, .2]))
    ndim = 2 if fam in ("star2", "box2") else (3 if fam != "any" else int(g.choice([2, 3])))
    shape = B.STAR if fam.startswith("star") else (B.BOX if fam.startswith("box")
                                                    else int(g.choice([B.STAR, B.BOX])))
    rmax = 4 if (shape == B.STAR or ndim == 2) else 3
    if fam == "box3":
        radius = 1
    elif fam == "any":
        radius = int(g.integers(0, rmax + 1))
    else:
        radius = int(g.integers(1, rmax + 1))
    dtype = str(g.choice(["f32", "f64"]))
    vec = 4 if dtype == "f32" else 2
    boundary = int(g.choice([B.ZERO, B.PERIODIC]))
    field = bool(g.random() < (0.5 if fam in ("box3", "any") else 0.0))
    channels = int(g.integers(1, 3))
    batch = channels * int(g.integers(1, 3)) if g.random() < 0.4 else 1
    steps = int(g.integers(0, 6))
    kind = int(g.choice([0, 1, 2], p=[.45, .4, .15]))
    if kind == 0:
        nx = vec * int(g.integers(1, 17))            # 16-byte vectors, ragged against tiles
    elif kind == 1:
        nx = vec * 64 * int(g.integers(1, 3))        # whole 64-lane row segments
    else:
        nx = int(g.integers(1, 70))                  # anything (generic if unaligned)
    if fam == "box3" and kind == 0:
        nx = vec * int(g.choice([2, 4, 8, 16, 32]))  # narrow rows the box packs per wavefront
    dims = (int(g.integers(1, 41)), nx) if ndim == 2 else \
        (int(g.integers(1, 25)), int(g.integers(1, 41)), nx)
    npts = B.stencil_num_points(shape, ndim, radius)
    # bound the oracle's work: points x offsets x steps
    while np.prod(dims) * batch * npts * max(steps, 1) > 3e7 and dims[0] > 1:
        dims = (max(1, dims[0] // 2),) + tuple(dims[1:])
    wl = replace(WORKLOADS["c4"], name="random%d" % seed, ndim=ndim, dims=tuple(dims),
                 batch=batch, channels=channels, dtype=dtype, shape=shape, radius=radius,
                 boundary=boundary, steps=steps, has_field=field)
    npdt = np.float32 if dtype == "f32" else np.float64
    lead = (batch,) if batch > 1 else ()
    x = g.uniform(-1, 1, lead + tuple(dims)).astype(npdt)
    w = g.uniform(-1, 1, (channels, npts))
    w = (w / np.abs(w).sum(axis=1, keepdims=True)).astype(npdt)
    k = g.uniform(0.5, 1.0, x.shape).astype(npdt) if field else None
    return wl, x, w, k


@pytest.mark.parametrize("seed", SEEDS)
def test_random_description(seed):
    wl, x, w, k = draw(seed)
    print("[case] random %d: ndim=%d shape=%d R=%d %s bnd=%d field=%s batch=%d ch=%d "
          "steps=%d dims=%s" % (seed, wl.ndim, wl.shape, wl.radius, wl.dtype, wl.boundary,
                                k is not None, wl.batch, wl.channels, wl.steps, wl.dims),
          flush=True)
    got, info = run_library(wl, x, w, k)
    print("[info] %s" % info, flush=True)
    report("random %d %s" % (seed, info), got, oracle_full(wl, x, w, k), tolerance(wl, x, k))


@pytest.mark.parametrize("seed", SEEDS[:60])
def test_random_description_forced_launch(seed):
    """The same draws with a forced launch configuration: one step per launch, a drawn grid
    scale (-2..2) and, for the one-step kernels that have two tiles, a drawn tile."""
    wl, x, w, k = draw(seed)
    g = np.random.default_rng(5000 + seed)
    desc = B.make_desc(wl.ndim, wl.dims, batch=wl.batch, channels=wl.channels,
                       dtype=B.F32 if wl.dtype == "f32" else B.F64, shape=wl.shape,
                       radius=wl.radius, boundary=wl.boundary, has_coeff_field=k is not None,
                       temporal_depth=1)
    plan = B.Plan(desc)
    kernel = plan.info().kernel.decode()
    plan.close()
    tiles = kernel in ("stencil_star_stream_kernel", "stencil_box3_stream_kernel")
    tile = int(g.integers(1, 3)) if tiles else 0
    gs = int(g.integers(-2, 3))
    print("[case] random %d forced: depth 1 tile %d grid_scale %d (%s)" % (seed, tile, gs,
                                                                         kernel), flush=True)
    got, info = run_library(wl, x, w, k, depth=1, tile=tile, grid_scale=gs)
    report("random %d forced %s" % (seed, info), got, oracle_full(wl, x, w, k),
           tolerance(wl, x, k))


@pytest.mark.parametrize("seed", SEEDS[:60])
def test_random_description_deepest_fusion(seed):
    """The same draws with the deepest temporal blocking the description allows (four steps
    per pass for fp32 radius-1 3D stars, three for fp64 ones, two for other 3D stars and 2D
    boxes)."""
    wl, x, w, k = draw(seed)
    desc = B.make_desc(wl.ndim, wl.dims, batch=wl.batch, channels=wl.channels,
                       dtype=B.F32 if wl.dtype == "f32" else B.F64, shape=wl.shape,
                       radius=wl.radius, boundary=wl.boundary, has_coeff_field=k is not None)
    depth = 1
    for d in (4, 3, 2):
        desc.temporal_depth = d
        try:
            B.Plan(desc).close()
            depth = d
            break
        except B.StencilError:
            continue
    print("[case] random %d deepest: depth %d" % (seed, depth), flush=True)
    got, info = run_library(wl, x, w, k, depth=depth)
    report("random %d deepest %s" % (seed, info), got, oracle_full(wl, x, w, k),
           tolerance(wl, x, k))


@pytest.mark.parametrize("seed", list(range(24)))
def test_random_deep_fusion(seed):
    """Radius-1 3D stars at the deepest fusion (four steps per pass in fp32, three in fp64)
    on drawn extents (1-30 planes, 1-45 rows, 1-20 vectors), batches with weight sets, both
    boundaries and 1-9 steps, every point against the oracle."""
    g = np.random.default_rng(7000 + seed)
    dtype = str(g.choice(["f32", "f64"]))
    vec = 4 if dtype == "f32" else 2
    dims = (int(g.integers(1, 31)), int(g.integers(1, 46)), vec * int(g.integers(1, 21)))
    channels = int(g.integers(1, 3))
    batch = channels * int(g.integers(1, 3)) if g.random() < 0.4 else 1
    wl = replace(WORKLOADS["c2"], name="deep%d" % seed, dims=dims, batch=batch,
                 channels=channels, dtype=dtype, boundary=int(g.choice([B.ZERO, B.PERIODIC])),
                 steps=int(g.integers(1, 10)))
    npdt = np.float32 if dtype == "f32" else np.float64
    x = g.uniform(-1, 1, ((batch,) if batch > 1 else ()) + dims).astype(npdt)
    w = g.uniform(-1, 1, (channels, wl.npoints))
    w = (w / np.abs(w).sum(axis=1, keepdims=True)).astype(npdt)
    depth = 4 if dtype == "f32" else 3
    print("[case] deep %d: %s bnd=%d batch=%d ch=%d steps=%d dims=%s depth=%d" % (
        seed, dtype, wl.boundary, batch, channels, wl.steps, dims, depth), flush=True)
    got, info = run_library(wl, x, w, depth=depth)
    assert info["kernel"] == "stencil_star_tbs_kernel", info
    report("deep %d %s" % (seed, info), got, oracle_full(wl, x, w), tolerance(wl, x))
