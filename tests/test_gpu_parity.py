"""GPU parity: the HIP library (through the C ABI) against the fp64 CPU oracle.

Reduced sizes (several tiles and ragged tails in every axis) are compared element by
element with the full oracle.  The full workload sizes are compared at every point too:
the oracle runs there in independent slabs or volumes on host threads
(``oracle/whole_grid.py``).
"""
import numpy as np
import pytest
import torch

from paper_2608_21157_amd import binding as B
from paper_2608_21157_amd import inputs
from paper_2608_21157_amd.inputs import WORKLOADS
from parity_util import dense_report, oracle_full, report, run_library, tolerance


pytestmark = pytest.mark.gpu

VARIANTS = [B.VARIANT_AUTO, B.VARIANT_GENERIC]

REDUCED = [
    ("c1", (256, 256), None, None),
    ("c1", (37, 61), None, None),
    ("c2", (40, 36, 72), None, None),
    ("c2", (33, 19, 20), None, 3),
    ("c3", (24, 40, 264), None, None),
    ("c3", (17, 23, 520), None, 1),
    ("c4", (20, 18, 520), None, None),
    ("c4", (9, 13, 256), None, None),
    ("c5", (20, 24, 128), 2, None),
    ("c5b", (12, 10, 128), 1, None),
    ("paper", (300, 260), None, 3),
]


def _case(name, dims, n, steps):
    wl = WORKLOADS[name].resized(dims, n=n, steps=steps)
    return wl, inputs.make(wl)


@pytest.mark.parametrize("variant", VARIANTS, ids=["auto", "generic"])
@pytest.mark.parametrize("name,dims,n,steps", REDUCED,
                         ids=["%s-%s" % (r[0], "x".join(map(str, r[1]))) for r in REDUCED])
def test_reduced_size_parity(name, dims, n, steps, variant):
    wl, (x, w, k) = _case(name, dims, n, steps)
    print("[case] %s dims=%s steps=%d variant=%d" % (name, dims, wl.steps, variant), flush=True)
    got, info = run_library(wl, x, w, k, variant=variant)
    ref = oracle_full(wl, x, w, k)
    report("%s %s %s" % (name, dims, info), got, ref, tolerance(wl, x, k))


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5", "c5b"])
def test_full_size_every_point(name):
    """Each workload at its full size, in the launch configuration the bench times (the
    planner's default plan), compared with the oracle at every point; the norm bound
    |S^s x| <= (max k * sum|w|)^s * max|x| is checked at every point as well."""
    wl = WORKLOADS[name]
    print("[case] full %s dims=%s batch=%d steps=%d" % (name, wl.dims, wl.batch, wl.steps),
          flush=True)
    x, w, k = inputs.make(wl)
    got, info = run_library(wl, x, w, k, as_f64=False)
    print("[info] %s" % info, flush=True)
    dense_report("full %s %s" % (name, info["kernel"]), wl, x, w, k, got, tolerance(wl, x, k))
    gain = float(np.abs(w.astype(np.float64)).sum(axis=1).max())
    if k is not None:
        gain *= float(k.max())
    bound = gain ** wl.steps * float(np.abs(x).max())
    assert float(np.abs(got).max()) <= bound * (1 + 1e-5) + tolerance(wl, x, k)


@pytest.mark.parametrize("steps", [0, 1, 2, 3, 4, 5])
@pytest.mark.parametrize("name", ["c2", "c3", "c4"])
def test_steps_and_ping_pong(name, steps):
    wl, (x, w, k) = _case(name, (14, 21, 264) if name != "c4" else (11, 9, 256), None, steps)
    got, _ = run_library(wl, x, w, k, steps=steps)
    ref = oracle_full(wl, x, w, k, steps=steps)
    report("%s steps=%d" % (name, steps), got, ref, tolerance(wl, x, k, steps))
    if steps == 0:
        assert np.array_equal(got, x.astype(np.float64))


TINY = [(1, 1, 1), (1, 2, 3), (2, 4, 9), (3, 1, 4), (5, 6, 7), (9, 3, 8)]


@pytest.mark.parametrize("dims", TINY)
@pytest.mark.parametrize("shape,R", [(B.STAR, 4), (B.BOX, 1), (B.BOX, 3), (B.STAR, 1)])
@pytest.mark.parametrize("boundary", [B.ZERO, B.PERIODIC])
def test_tiny_grids(dims, shape, R, boundary):
    g = np.random.default_rng(3)
    wl = WORKLOADS["c4"].resized(dims)
    from dataclasses import replace
    wl = replace(wl, shape=shape, radius=R, boundary=boundary, steps=2, has_field=False)
    x = g.uniform(-1, 1, dims).astype(np.float32)
    w = g.uniform(-1, 1, (1, wl.npoints))
    w = (w / np.abs(w).sum()).astype(np.float32)
    got, _ = run_library(wl, x, w)
    ref = oracle_full(wl, x, w)
    report("tiny %s shape=%d R=%d bnd=%d" % (dims, shape, R, boundary), got, ref,
           tolerance(wl, x))


def test_input_untouched_and_guard_band():
    """`in` is not modified; NaN guard cells around `out` stay NaN."""
    wl, (x, w, k) = _case("c4", (10, 12, 256), None, None)
    dev = torch.device("cuda:0")
    xt = torch.from_numpy(x).to(dev)
    kt = torch.from_numpy(k).to(dev)
    n = x.size
    pad = 4096
    buf = torch.full((n + 2 * pad,), float("nan"), dtype=xt.dtype, device=dev)
    y = buf[pad:pad + n].view(x.shape)
    B.apply(xt, y, w, shape=wl.shape, radius=wl.radius, boundary=wl.boundary, steps=1,
            field=kt, ndim=3)
    torch.cuda.synchronize()
    assert torch.isnan(buf[:pad]).all() and torch.isnan(buf[pad + n:]).all()
    assert np.array_equal(xt.cpu().numpy(), x)
    ref = oracle_full(wl, x, w, k)
    report("guard", y.cpu().numpy().astype(np.float64), ref, tolerance(wl, x, k))


def test_misaligned_pointers_fall_back():
    """Pointers off the 16-byte grid run a scalar kernel and still match."""
    wl, (x, w, k) = _case("c3", (12, 14, 264), None, 2)
    dev = torch.device("cuda:0")
    n = x.size
    bx = torch.zeros(n + 1, dtype=torch.float32, device=dev)
    by = torch.zeros(n + 1, dtype=torch.float32, device=dev)
    xt = bx[1:].view(x.shape)
    xt.copy_(torch.from_numpy(x).to(dev))
    yt = by[1:].view(x.shape)
    B.apply(xt, yt, w, shape=wl.shape, radius=wl.radius, boundary=wl.boundary, steps=2, ndim=3)
    torch.cuda.synchronize()
    ref = oracle_full(wl, x, w, k, steps=2)
    report("misaligned", yt.cpu().numpy().astype(np.float64), ref, tolerance(wl, x, steps=2))


def test_plan_reuse_with_changing_weights():
    """One plan, two weight sets in a row on one stream (distinct arrays, then one array
    changed in place): each call sees its own weights."""
    wl, (x, w, k) = _case("c4", (8, 9, 256), None, None)
    dev = torch.device("cuda:0")
    xt = torch.from_numpy(x).to(dev)
    kt = torch.from_numpy(k).to(dev)
    desc = B.make_desc(3, x.shape, shape=wl.shape, radius=1, boundary=wl.boundary,
                       has_coeff_field=True)
    plan = B.Plan(desc)
    try:
        outs = []
        w2 = (-w[:, ::-1]).copy()
        for ww in (w, w2, w):
            y = torch.empty_like(xt)
            plan.run(xt, y, ww, steps=1, field=kt)
            outs.append((ww, y))
        # one array object whose values change in place between calls
        wm = w.copy()
        for ww in (w, w2):
            wm[...] = ww
            y = torch.empty_like(xt)
            plan.run(xt, y, wm, steps=1, field=kt)  # copies the weights before returning
            outs.append((ww, y))
        torch.cuda.synchronize()
        for ww, y in outs:
            ref = oracle_full(wl, x, ww, k)
            report("reuse", y.cpu().numpy().astype(np.float64), ref, tolerance(wl, x, k))
    finally:
        plan.close()


def test_nondefault_stream():
    wl, (x, w, k) = _case("c3", (16, 20, 264), None, 3)
    s = torch.cuda.Stream()
    got, _ = run_library(wl, x, w, k, stream=s)
    ref = oracle_full(wl, x, w, k)
    report("stream", got, ref, tolerance(wl, x, k))


def test_run_without_a_stream_follows_torchs_current_stream():
    """Plan.run with no stream launches on torch's current stream, resolved again on every
    call: two side streams are made current in turn, each first spins (torch.cuda._sleep)
    and then writes the input, so a launch on any other stream would read the input
    before it is written.  Both calls must match the oracle."""
    wl, (x, w, k) = _case("c3", (16, 20, 264), None, 2)
    ref = oracle_full(wl, x, w, k)
    src = torch.from_numpy(x).to(torch.device("cuda:0"))
    torch.cuda.synchronize()
    plan = B.Plan(B.make_desc(wl.ndim, wl.dims, shape=wl.shape, radius=wl.radius,
                              boundary=wl.boundary))
    try:
        for round_ in range(2):
            side = torch.cuda.Stream()
            with torch.cuda.stream(side):
                xt = torch.zeros_like(src)
                yt = torch.full_like(src, float("nan"))
                torch.cuda._sleep(20_000_000)
                xt.copy_(src)
                plan.run(xt, yt, w, steps=wl.steps)
            side.synchronize()
            report("current stream %d" % round_, yt.cpu().numpy().astype(np.float64), ref,
                   tolerance(wl, x, k))
    finally:
        plan.close()


def test_variants_agree():
    """Every variant the planner can force gives the oracle's result on the same input."""
    wl, (x, w, k) = _case("c4", (16, 20, 512), None, None)
    ref = oracle_full(wl, x, w, k)
    for variant in (B.VARIANT_GENERIC, B.VARIANT_AUTO):
        got, info = run_library(wl, x, w, k, variant=variant)
        report("variant %s" % info, got, ref, tolerance(wl, x, k))


STAR_CASES = [(R, dt, bnd) for R in (1, 2, 3, 4) for dt in ("f32", "f64")
              for bnd in (B.ZERO, B.PERIODIC)]


@pytest.mark.parametrize("R,dt,bnd", STAR_CASES,
                         ids=["R%d-%s-%s" % (c[0], c[1], "zero" if c[2] == 0 else "per")
                              for c in STAR_CASES])
@pytest.mark.parametrize("depth", [1, 2, 0], ids=["depth1", "depth2", "auto"])
def test_star_radius_dtype_boundary_depth(R, dt, bnd, depth):
    """3D stars of every radius, fp32 and fp64, both boundaries, one launch per step,
    steps fused two at a time, or the planner's choice; ragged extents in every axis,
    3 steps (one fused pair plus a single step)."""
    from dataclasses import replace
    g = np.random.default_rng(100 + R)
    dims = (23, 37, 72) if dt == "f32" else (21, 35, 40)
    wl = replace(WORKLOADS["c3"].resized(dims, steps=3), radius=R, boundary=bnd, dtype=dt)
    npdt = np.float32 if dt == "f32" else np.float64
    x = g.uniform(-1, 1, dims).astype(npdt)
    w = g.uniform(-1, 1, (1, wl.npoints))
    w = (w / np.abs(w).sum()).astype(npdt)
    got, info = run_library(wl, x, w, depth=depth)
    ref = oracle_full(wl, x, w)
    report("star R=%d %s bnd=%d %s" % (R, dt, bnd, info), got, ref, tolerance(wl, x))


def test_fused_steps_match_single_steps():
    """Two steps in one fused pass agree with two single-step launches (both against the
    oracle, and with each other to rounding)."""
    wl, (x, w, k) = _case("c3", (40, 33, 136), None, 2)
    fused, i2 = run_library(wl, x, w, depth=2)
    single, i1 = run_library(wl, x, w, depth=1)
    assert i2["depth"] == 2 and i1["depth"] == 1
    ref = oracle_full(wl, x, w)
    report("fused", fused, ref, tolerance(wl, x))
    report("single", single, ref, tolerance(wl, x))
    assert np.abs(fused - single).max() <= 2 * tolerance(wl, x)


BOX2_CASES = [(R, dt, bnd) for R in (1, 2, 3, 4) for dt in ("f32", "f64")
              for bnd in (B.ZERO, B.PERIODIC)]


@pytest.mark.parametrize("R,dt,bnd", BOX2_CASES,
                         ids=["R%d-%s-%s" % (c[0], c[1], "zero" if c[2] == 0 else "per")
                              for c in BOX2_CASES])
@pytest.mark.parametrize("nx", [512, 32], ids=["wide", "narrow"])
@pytest.mark.parametrize("depth", [1, 0], ids=["depth1", "auto"])
def test_box2d_radius_dtype_boundary(R, dt, bnd, nx, depth):
    """2D boxes (the paper's operator family): every radius up to 4, fp32 and fp64, both
    boundaries, rows that span several 64-lane segments or several rows per wavefront,
    a ragged row count and 3 steps, batch 3 with 2 weight sets."""
    from dataclasses import replace
    g = np.random.default_rng(200 + R)
    wl = replace(WORKLOADS["paper"].resized((131, nx), steps=3), radius=R, boundary=bnd,
                 dtype=dt, batch=3, channels=2)
    npdt = np.float32 if dt == "f32" else np.float64
    x = g.uniform(-1, 1, (3, 131, nx)).astype(npdt)
    w = g.uniform(-1, 1, (2, wl.npoints))
    w = (w / np.abs(w).sum(axis=1, keepdims=True)).astype(npdt)
    got, info = run_library(wl, x, w, depth=depth)
    assert info["kernel"] in ("stencil_box2_stream_kernel", "stencil_box2_tb2_kernel"), info
    ref = oracle_full(wl, x, w)
    report("box2d R=%d %s bnd=%d nx=%d %s" % (R, dt, bnd, nx, info), got, ref,
           tolerance(wl, x))


def test_paper_workload_full_size_every_point():
    """The paper's own case: 2D 49-point box, radius 3, 10240 x 10240 fp64, zero padding,
    three steps of the iteration (a fused pass and a one-step pass through the ping-pong
    grid), every point against the oracle."""
    wl = WORKLOADS["paper"].resized((10240, 10240), steps=3)
    x, w, _ = inputs.make(wl)
    got, info = run_library(wl, x, w, as_f64=False)
    print("[info] %s" % info, flush=True)
    assert info["kernel"] in ("stencil_box2_stream_kernel", "stencil_box2_tb2_kernel")
    dense_report("paper full", wl, x, w, None, got, tolerance(wl, x))


def test_2d_image_beyond_the_streaming_limit_runs_generic():
    """A 2D fp64 image over 1 GiB (11600 x 11600) exceeds the 32-bit byte offsets of the
    2D box kernels: the planner falls back to the generic kernel, which indexes in 64 bits.
    Two steps (ping-pong through the plan's scratch), every point against the oracle."""
    wl = WORKLOADS["paper"].resized((11600, 11600), steps=2)
    assert wl.points_per_step * wl.itemsize > (1 << 30)
    x, w, _ = inputs.make(wl)
    got, info = run_library(wl, x, w, as_f64=False)
    print("[info] %s" % info, flush=True)
    assert info["kernel"] == "stencil_generic_kernel"
    dense_report("2D beyond the streaming limit", wl, x, w, None, got, tolerance(wl, x))


@pytest.mark.parametrize("depth", [2, 1], ids=["fused", "one-step"])
def test_maximum_size_star_1024_cubed(depth):
    """The largest grid the tests drive: 1024^3 fp32 (2^30 points, 4 GiB per grid, eight
    times the headline volume), the 25-point radius-4 star over 2 steps, fused or one step
    per launch, every point against the oracle."""
    dims = (1024, 1024, 1024)
    wl = WORKLOADS["c3"].resized(dims, steps=2)
    _, w, _ = inputs.make(WORKLOADS["c3"].resized((8, 8, 8)))  # the c3 weights
    g = np.random.default_rng(77)
    x = g.random(dims, dtype=np.float32)
    x *= 2
    x -= 1
    print("[case] max size %s depth=%d" % (dims, depth), flush=True)
    xt = torch.from_numpy(x).to("cuda:0")
    yt = torch.empty_like(xt)
    plan = B.Plan(B.make_desc(3, dims, shape=B.STAR, radius=4, temporal_depth=depth))
    try:
        assert plan.info().temporal_depth == depth
        plan.run(xt, yt, w, steps=wl.steps)
        torch.cuda.synchronize()
    finally:
        plan.close()
    got = yt.cpu().numpy()
    del xt, yt
    torch.cuda.empty_cache()
    dense_report("max size depth %d" % depth, wl, x, w, None, got, tolerance(wl, x))


GUARD_CASES = [
    # name, dims, steps: star fused + trailing single step, 2D box fused, 2D star, box3
    ("c3", (18, 40, 136), 3),
    ("paper", (70, 260), 3),
    ("c1", (40, 68), 2),
    ("c5", (10, 12, 128), 2),
]


@pytest.mark.parametrize("name,dims,steps", GUARD_CASES, ids=[c[0] for c in GUARD_CASES])
def test_guard_band_and_input_every_family(name, dims, steps):
    """Multi-launch calls (ping-pong through the plan's grid, fused passes) write only
    inside `out` (NaN canaries on both sides stay NaN) and never write `in`."""
    n = 1 if name == "c5" else None
    wl, (x, w, k) = _case(name, dims, n, steps)
    dev = torch.device("cuda:0")
    xt = torch.from_numpy(x).to(dev)
    pad = 8192
    buf = torch.full((x.size + 2 * pad,), float("nan"), dtype=xt.dtype, device=dev)
    y = buf[pad:pad + x.size].view(x.shape)
    lead = x.shape[: x.ndim - wl.ndim]
    batch = int(np.prod(lead)) if len(lead) else 1
    desc = B.make_desc(wl.ndim, wl.dims, batch=batch, channels=wl.channels,
                       dtype=B.F32 if wl.dtype == "f32" else B.F64, shape=wl.shape,
                       radius=wl.radius, boundary=wl.boundary)
    plan = B.Plan(desc)
    try:
        print("[case] guard %s %s steps=%d kernel=%s depth=%d" % (
            name, dims, steps, plan.info().kernel.decode(), plan.info().temporal_depth),
            flush=True)
        plan.run(xt, y, w, steps=steps)
        torch.cuda.synchronize()
    finally:
        plan.close()
    assert torch.isnan(buf[:pad]).all() and torch.isnan(buf[pad + x.size:]).all()
    assert np.array_equal(xt.cpu().numpy(), x)
    report("guard %s" % name, y.cpu().numpy().astype(np.float64), oracle_full(wl, x, w),
           tolerance(wl, x))


RAGGED = [
    # streaming families on the extents 17, 63, 65, 257 (x a multiple of 16 bytes)
    ("c3", (17, 63, 260), 3),
    ("c3", (65, 17, 68), 2),
    ("c2", (63, 65, 20), 3),
    ("c4", (17, 65, 256), None),
    ("paper", (257, 260), 3),
    ("paper", (63, 1028), 2),
]


@pytest.mark.parametrize("name,dims,steps", RAGGED,
                         ids=["%s-%s" % (r[0], "x".join(map(str, r[1]))) for r in RAGGED])
def test_ragged_extents(name, dims, steps):
    wl, (x, w, k) = _case(name, dims, None, steps)
    got, info = run_library(wl, x, w, k)
    print("[info] %s" % info, flush=True)
    report("ragged %s %s" % (name, dims), got, oracle_full(wl, x, w, k), tolerance(wl, x, k))


BOX3_CHUNKS = [("c4", 2), ("c4", 1), ("c5", 2), ("c5b", 1)]


@pytest.mark.parametrize("name,gs", BOX3_CHUNKS, ids=["%s-s%d" % c for c in BOX3_CHUNKS])
def test_box3_z_chunks_both_directions(name, gs):
    """The 27-point box streams even z chunks upwards and odd ones downwards (mirrored z
    weights).  37 planes in chunks of 4 (grid scale 2: ten chunks, the last one plane) or
    of 8 (grid scale 1: five chunks, the last five planes); periodic with a field (c4) and
    zero boundary with per-channel weights (c5, c5b); every point against the oracle."""
    wl, (x, w, k) = _case(name, (37, 10, 256 if name == "c4" else 128),
                          None if name == "c4" else 1, None)
    print("[case] box3 chunks %s dims=%s grid_scale=%d" % (name, wl.dims, gs), flush=True)
    got, info = run_library(wl, x, w, k, grid_scale=gs)
    assert info["kernel"] == "stencil_box3_stream_kernel", info
    report("box3 chunks %s s%d %s" % (name, gs, info), got, oracle_full(wl, x, w, k),
           tolerance(wl, x, k))


@pytest.mark.parametrize("gs", [-1, 0, 1], ids=["s-1", "s0", "s1"])
def test_star_fused_z_chunks(gs):
    """The fused star's z chunking at radius 1 on 203 x 256^2, two steps: grid scale 0 is
    one workgroup per CU in 26-plane chunks (a round of two per CU would give 13-plane
    chunks), +1 that former round, -1 51-plane chunks; the last chunk of each is short and
    odd chunks stream downwards.  Every point against the oracle."""
    wl, (x, w, k) = _case("c2", (203, 256, 256), None, 2)
    print("[case] star fused z chunks dims=%s grid_scale=%d" % (wl.dims, gs), flush=True)
    got, info = run_library(wl, x, w, k, grid_scale=gs)
    assert info["kernel"] == "stencil_star_tb2_kernel", info
    report("star chunks s%d %s" % (gs, info), got, oracle_full(wl, x, w, k),
           tolerance(wl, x, k))


RADIUS0 = [(B.STAR, 3, B.ZERO, False), (B.BOX, 3, B.PERIODIC, True),
           (B.BOX, 2, B.ZERO, False), (B.STAR, 2, B.PERIODIC, False)]


@pytest.mark.parametrize("shape,ndim,boundary,field", RADIUS0,
                         ids=["%s%dd-%s%s" % ("star" if c[0] == B.STAR else "box", c[1],
                                              "zero" if c[2] == B.ZERO else "per",
                                              "-field" if c[3] else "") for c in RADIUS0])
def test_radius_zero(shape, ndim, boundary, field):
    """Radius 0, the degenerate stencil (the centre only): each step scales every point by
    k w0.  Three steps over four volumes with two weight sets, every point against the
    oracle (the planner runs the generic kernel here)."""
    from dataclasses import replace
    dims = (6, 10, 36) if ndim == 3 else (20, 36)
    wl = replace(WORKLOADS["c4"].resized((6, 10, 36)), ndim=ndim, dims=dims, shape=shape,
                 radius=0, boundary=boundary, steps=3, has_field=field, channels=2)
    g = np.random.default_rng(41)
    x = g.uniform(-1, 1, (4,) + dims).astype(np.float32)
    w = g.uniform(-1, 1, (2, 1)).astype(np.float32)
    k = g.uniform(0.5, 1.0, x.shape).astype(np.float32) if field else None
    print("[case] radius 0 shape=%d ndim=%d boundary=%d field=%s" % (shape, ndim, boundary,
                                                                    field), flush=True)
    got, info = run_library(wl, x, w, k)
    report("radius 0 %s" % info, got, oracle_full(wl, x, w, k), tolerance(wl, x, k))


TBS_CASES = [(dt, d, n, bnd) for dt, d, steps in (("f32", 4, (4, 5, 6, 7, 9)),
                                                  ("f32", 3, (3, 5)), ("f64", 3, (3, 4, 5, 7)))
             for n in steps for bnd in (B.ZERO, B.PERIODIC)]


@pytest.mark.parametrize("dt,depth,steps,bnd", TBS_CASES,
                         ids=["%s-d%d-s%d-%s" % (c[0], c[1], c[2],
                                                 "zero" if c[3] == B.ZERO else "per")
                              for c in TBS_CASES])
def test_star_four_steps_per_pass(dt, depth, steps, bnd):
    """Radius-1 3D stars with three or four steps fused per pass (fp32) or three (fp64),
    trailing passes of one or two steps for the remainder, ragged extents in every axis,
    every point."""
    from dataclasses import replace
    g = np.random.default_rng(200 + 10 * depth + steps)
    npdt = np.float32 if dt == "f32" else np.float64
    for dims in (((23, 37, 72), (9, 3, 40)) if dt == "f32" else ((21, 35, 38), (9, 3, 20))):
        wl = replace(WORKLOADS["c2"].resized(dims, steps=steps), boundary=bnd, dtype=dt)
        x = g.uniform(-1, 1, dims).astype(npdt)
        w = g.uniform(-1, 1, (1, wl.npoints))
        w = (w / np.abs(w).sum()).astype(npdt)
        print("[case] tbs %s depth=%d steps=%d bnd=%d dims=%s" % (dt, depth, steps, bnd, dims),
              flush=True)
        got, info = run_library(wl, x, w, depth=depth)
        assert info["kernel"] == "stencil_star_tbs_kernel" and info["depth"] == depth, info
        report("tbs %s %s" % (dims, info), got, oracle_full(wl, x, w), tolerance(wl, x))


def test_star_four_steps_per_pass_512_cubed():
    """The planner's choice for an fp32 radius-1 star beyond the Infinity Cache: four
    steps per pass.  512^3, 10 steps (4 + 4 + 2), every point against the oracle."""
    wl = WORKLOADS["c2_512"]
    x, w, _ = inputs.make(wl)
    print("[case] tbs 512^3 steps=%d" % wl.steps, flush=True)
    got, info = run_library(wl, x, w, as_f64=False)
    assert info["kernel"] == "stencil_star_tbs_kernel" and info["depth"] == 4, info
    dense_report("tbs 512^3", wl, x, w, None, got, tolerance(wl, x))
