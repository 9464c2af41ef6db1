"""HIP graph capture of stencil_apply (torch.cuda.graph over the C ABI).

Once a plan has run (its device buffers exist and its weights are uploaded) and its
weights stay the same, a call enqueues kernel launches only, so a caller can capture calls
in a HIP graph and replay them.  Each replay is checked against the eager result of the
same input (the same kernels in the same order give identical bits) and against the
oracle.  The input is rewritten between replays, with eager work and synchronisation in
between, so every replay must read the buffers as they are at replay time.
"""
import numpy as np
import pytest
import torch

from paper_2608_21157_amd import binding as B
from paper_2608_21157_amd import inputs
from paper_2608_21157_amd.inputs import WORKLOADS
from parity_util import oracle_full, report, tolerance

pytestmark = pytest.mark.gpu

CASES = [
    ("c1", (256, 256), None),      # one launch
    ("c3", (20, 24, 264), 4),      # two fused launches through the plan's ping-pong grid
    ("c4", (12, 10, 520), None),   # periodic, coefficient field
    ("paper", (300, 260), 3),      # fused pass plus a one-step launch
]


@pytest.mark.parametrize("name,dims,steps", CASES,
                         ids=["%s-%s" % (c[0], "x".join(map(str, c[1]))) for c in CASES])
def test_graph_replays_match_eager(name, dims, steps):
    wl = WORKLOADS[name].resized(dims, steps=steps)
    x, w, k = inputs.make(wl)
    print("[case] graph %s dims=%s steps=%d" % (name, dims, wl.steps), flush=True)
    dev = torch.device("cuda:0")
    xt = torch.from_numpy(x).to(dev)
    kt = None if k is None else torch.from_numpy(k).to(dev)
    y_eager = torch.empty_like(xt)
    y_graph = torch.full_like(xt, float("nan"))
    desc = B.make_desc(wl.ndim, wl.dims, batch=wl.batch, channels=wl.channels,
                       dtype=B.F32 if wl.dtype == "f32" else B.F64, shape=wl.shape,
                       radius=wl.radius, boundary=wl.boundary, has_coeff_field=kt is not None)
    plan = B.Plan(desc)
    s = torch.cuda.Stream()
    try:
        plan.run(xt, y_eager, w, steps=wl.steps, field=kt, stream=s)  # first use
        s.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            plan.run(xt, y_graph, w, steps=wl.steps, field=kt)
        plan._stream = s
        g2 = np.random.default_rng(11)
        for rep in range(3):
            xr = x if rep == 0 else (x * g2.uniform(0.5, 1.0)).astype(x.dtype)
            xt.copy_(torch.from_numpy(xr))
            y_graph.fill_(float("nan"))
            torch.cuda.synchronize()
            with torch.cuda.stream(s):
                g.replay()
            s.synchronize()
            got = y_graph.cpu().numpy()
            plan.run(xt, y_eager, w, steps=wl.steps, field=kt, stream=s)  # eager, same input
            s.synchronize()
            assert np.array_equal(got, y_eager.cpu().numpy()), "replay %d differs" % rep
            report("graph %s replay %d" % (name, rep), got.astype(np.float64),
                   oracle_full(wl, xr, w, k), tolerance(wl, xr, k))
        del g
    finally:
        plan.close()
