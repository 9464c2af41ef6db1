"""Independent plans used at the same time: each on its own stream, interleaved from one
host thread, and from two host threads at once (the binding releases the GIL during each
library call, so the calls really overlap).  A plan holds all of its mutable state (its
buffers, its weights, its launch choice); the library's only shared state is the
thread-local error string and the per-kernel occupancy counts computed once.  Every
result is compared with the oracle."""
import threading

import numpy as np
import pytest
import torch

from paper_2608_21157_amd import binding as B
from paper_2608_21157_amd import inputs
from paper_2608_21157_amd.inputs import WORKLOADS
from parity_util import oracle_full, report, tolerance

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
CASES = [("c3", (20, 24, 264), 4), ("c4", (12, 10, 520), None), ("paper", (130, 260), 3)]


class Job:
    def __init__(self, name, dims, steps):
        self.wl = WORKLOADS[name].resized(dims, steps=steps)
        self.x, self.w, self.k = inputs.make(self.wl)
        self.xt = torch.from_numpy(self.x).to(DEV)
        self.kt = None if self.k is None else torch.from_numpy(self.k).to(DEV)
        self.yt = torch.empty_like(self.xt)
        wl = self.wl
        self.plan = B.Plan(B.make_desc(wl.ndim, wl.dims, batch=wl.batch, channels=wl.channels,
                                       dtype=B.F32 if wl.dtype == "f32" else B.F64,
                                       shape=wl.shape, radius=wl.radius, boundary=wl.boundary,
                                       has_coeff_field=self.kt is not None))
        self.stream = torch.cuda.Stream()
        torch.cuda.synchronize()

    def call(self):
        self.plan.run(self.xt, self.yt, self.w, steps=self.wl.steps, field=self.kt,
                      stream=self.stream)

    def check(self, label):
        self.stream.synchronize()
        report("%s %s" % (label, self.wl.name), self.yt.cpu().numpy().astype(np.float64),
               oracle_full(self.wl, self.x, self.w, self.k),
               tolerance(self.wl, self.x, self.k))

    def close(self):
        self.plan.close()


def test_plans_on_separate_streams_interleaved():
    jobs = [Job(*c) for c in CASES]
    try:
        for _ in range(10):
            for j in jobs:
                j.call()
        for j in jobs:
            j.check("interleaved")
    finally:
        for j in jobs:
            j.close()


def test_plans_from_two_host_threads():
    jobs = [Job(*c) for c in CASES[:2]]
    errors = []

    def work(j):
        try:
            for _ in range(20):
                j.call()
            j.stream.synchronize()
        except Exception as e:  # reported by the main thread
            errors.append(e)

    try:
        threads = [threading.Thread(target=work, args=(j,)) for j in jobs]
        for t in threads:
            t.start()
        for t in threads:
            t.join(timeout=60)
        assert not any(t.is_alive() for t in threads), "a host thread did not finish"
        assert not errors, errors
        for j in jobs:
            j.check("threads")
    finally:
        for j in jobs:
            j.close()
