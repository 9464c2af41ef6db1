"""stencil_apply_noalloc through the C ABI against stencil_apply on the same inputs.

Each case makes two allocation-free calls in a row on one stream, with no
synchronisation between them, the second on a smaller grid with other weights (both
share the GPU's static scratch), then compares each result with stencil_apply's (same
kernels and launch configuration, so the results must be identical) and, where the
oracle is quick, with the oracle.  The cases cover multi-launch calls whose intermediate
grid lives in the scratch (up to its 64 MiB limit), the 3D box with a coefficient field,
the paper's 2D fp64 box, the batched conv form with 32 weight sets, a single-launch call
on a grid far larger than the scratch, the refusal of a call that needs a larger
intermediate grid, and that the calls take no device memory.
"""
import numpy as np
import pytest
import torch

from paper_2608_21157_amd import binding as B
from paper_2608_21157_amd import inputs
from paper_2608_21157_amd.inputs import WORKLOADS
from parity_util import oracle_full, report, tolerance

pytestmark = pytest.mark.gpu


def _plan(wl, batch):
    return B.Plan(B.make_desc(wl.ndim, wl.dims, batch=batch, channels=wl.channels,
                              dtype=B.F32 if wl.dtype == "f32" else B.F64, shape=wl.shape,
                              radius=wl.radius, boundary=wl.boundary,
                              has_coeff_field=wl.has_field))


class Case:
    """One call's inputs on the GPU and both entry points' outputs."""

    def __init__(self, name, dims, n=None, steps=None, reweight=None):
        self.wl = WORKLOADS[name].resized(dims, n=n, steps=steps)
        self.x, self.w, self.k = inputs.make(self.wl)
        if reweight is not None:  # other weights than the recipe's, of the same form
            g = np.random.default_rng(reweight)
            w = g.uniform(-1, 1, self.w.shape)
            self.w = (w / np.abs(w).sum(axis=1, keepdims=True)).astype(self.w.dtype)
        dev = torch.device("cuda:0")
        self.xt = torch.from_numpy(self.x).to(dev)
        self.kt = None if self.k is None else torch.from_numpy(self.k).to(dev)
        self.y_noalloc = torch.full_like(self.xt, float("nan"))
        self.y_apply = torch.full_like(self.xt, float("nan"))
        lead = self.x.shape[: self.x.ndim - self.wl.ndim]
        self.batch = int(np.prod(lead)) if len(lead) else 1
        self.plan_n = _plan(self.wl, self.batch)   # used only by the allocation-free call
        self.plan_a = _plan(self.wl, self.batch)
        torch.cuda.synchronize()

    def noalloc(self, stream):
        B.stencil_apply_noalloc(self.plan_n.handle, self.xt.data_ptr(),
                                self.y_noalloc.data_ptr(), self.wl.dims, self.w,
                                None if self.kt is None else self.kt.data_ptr(),
                                self.wl.radius, self.wl.boundary, self.wl.steps,
                                stream.cuda_stream)

    def apply(self, stream):
        B.stencil_apply(self.plan_a.handle, self.xt.data_ptr(), self.y_apply.data_ptr(),
                        self.wl.dims, self.w, None if self.kt is None else self.kt.data_ptr(),
                        self.wl.radius, self.wl.boundary, self.wl.steps, stream.cuda_stream)

    def check(self, label, with_oracle=True):
        assert torch.equal(self.y_noalloc, self.y_apply), "%s: results differ" % label
        got = self.y_noalloc.cpu().numpy().astype(np.float64)
        assert np.isfinite(got).all()
        if with_oracle:
            report("noalloc %s" % label, got, oracle_full(self.wl, self.x, self.w, self.k),
                   tolerance(self.wl, self.x, self.k))

    def close(self):
        self.plan_n.close()
        self.plan_a.close()


PAIRS = [
    # (first call, second smaller call with other weights)
    (("c2", (256, 256, 256), None, 10), ("c2", (40, 36, 72), None, 3)),
    (("c4", (20, 18, 520), None, 1), ("c4", (9, 13, 256), None, 2)),
    (("paper", (300, 260), None, 5), ("paper", (70, 260), None, 3)),
    (("c5", (20, 24, 128), 2, 2), ("c5", (10, 12, 128), 1, 1)),
    (("c3", (512, 512, 512), None, 2), ("c3", (24, 40, 264), None, 4)),
]


@pytest.mark.parametrize("first,second", PAIRS, ids=[p[0][0] for p in PAIRS])
def test_two_calls_in_a_row_match_stencil_apply(first, second):
    print("[case] noalloc %s then %s" % (first, second), flush=True)
    a = Case(*first)
    b = Case(*second, reweight=17)
    s = torch.cuda.Stream()
    try:
        a.noalloc(s)
        b.noalloc(s)          # same stream, no synchronisation in between
        a.apply(s)
        b.apply(s)
        s.synchronize()
        big = a.x.size * max(a.wl.steps, 1) > 5e7
        a.check("%s %s steps=%d" % (first[0], a.wl.dims, a.wl.steps), with_oracle=not big)
        b.check("%s %s steps=%d" % (second[0], b.wl.dims, b.wl.steps))
    finally:
        a.close()
        b.close()


def test_weights_changing_between_calls():
    """Calls in a row on one stream whose weights repeat, change and change back (the
    library skips the upload when the device already holds the same bytes), across two
    plans of different sizes: every result matches stencil_apply's with its weights."""
    a = Case("c2", (24, 20, 64), steps=3)
    b = Case("c2", (16, 12, 32), steps=2)
    g = np.random.default_rng(5)
    w_other = g.uniform(-1, 1, a.w.shape)
    w_other = (w_other / np.abs(w_other).sum()).astype(a.w.dtype)
    s = torch.cuda.Stream()
    outs = []
    try:
        for case, w in ((a, a.w), (a, a.w), (b, a.w), (a, w_other), (b, w_other), (a, a.w)):
            case.w = w
            case.noalloc(s)
            case.apply(s)
            s.synchronize()
            assert torch.equal(case.y_noalloc, case.y_apply)
            outs.append(case.y_noalloc.clone())
        # the calls with the first weights agree with each other, the others differ
        assert torch.equal(outs[0], outs[1]) and torch.equal(outs[0], outs[5])
        assert not torch.equal(outs[0], outs[3])
        a.check("weights repeated and changed")
    finally:
        a.close()
        b.close()


def test_call_beyond_the_scratch_is_refused_and_writes_nothing():
    """The 27-point box on 512^3 fp32 over 2 steps (two launches) needs a 512 MiB
    intermediate grid: refused on the host, and `out` is left as it was."""
    c = Case("c4", (512, 512, 512), steps=2)
    s = torch.cuda.Stream()
    try:
        with pytest.raises(B.StencilError) as err:
            c.noalloc(s)
        assert err.value.status == B.ERR_UNSUPPORTED
        assert "intermediate grid" in str(err.value)
        s.synchronize()
        assert bool(torch.isnan(c.y_noalloc).all())
    finally:
        c.close()


def test_calls_take_no_device_memory():
    """After a first call (which finds the scratch), further calls, multi-launch ones
    included, leave the device's free memory where it was."""
    c = Case("c2", (64, 64, 128), steps=7)
    d = Case("c4", (16, 16, 256), steps=3)
    s = torch.cuda.Stream()
    try:
        c.noalloc(s)
        s.synchronize()
        free0, _ = torch.cuda.mem_get_info()
        for _ in range(3):
            c.noalloc(s)
            d.noalloc(s)
        s.synchronize()
        free1, _ = torch.cuda.mem_get_info()
        assert free1 == free0, "free device memory changed by %d bytes" % (free0 - free1)
        c.apply(s)
        d.apply(s)
        s.synchronize()
        c.check("memory c2")
        d.check("memory c4")
    finally:
        c.close()
        d.close()
