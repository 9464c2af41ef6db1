#!/usr/bin/env python3
"""Throughput of the MI355X stencil library on its headline workload, one GPU.

A step is one ``stencil_apply`` of the headline workload: the 25-point radius-4 star
(8th-order Laplacian weights) on a 512^3 fp32 grid, zero boundary, 4 stencil steps per
call, inputs already resident in HBM.  The metric is stencil points per second
(Gpoints/s = 512^3 * 4 / time per call) with the achieved HBM bandwidth of the dominant
kernel against the compulsory-traffic roofline (each point read once and written once
per stencil step: 8 bytes per point-step in fp32).

The headline value is K back-to-back calls after W warm-up calls.  Before those, the
headline kernel itself runs for a fixed time (``spin_up``): a stencil kernel reaches its
steady speed only after about 20 calls of itself, whatever ran before, so the value does
not depend on W.

Prints one JSON line on stdout; progress goes to stderr.  Besides the headline (with an
HBM roofline object and its flop-side counterpart) it reports:
  * per workload (2D 5-point, 3D 7-point x10, the headline, 27-point box with a
    coefficient field (periodic), depthwise 3x3x3 conv form in fp32 and fp64, and the
    paper's own 2D radius-3 fp64 box): back-to-back timing, and the paper's protocol --
    3 warm-up runs, then 100 timed runs, each after the caches are flushed, graded by
    the median, with the minimum reported;
  * per workload, the default plan's own output checked against the fp64 CPU oracle at
    every point of the full-size grid (the oracle's wall time, threads and error);
  * the oracle timed single-threaded on a bounded slab of the headline input
    (``cpu_baseline``);
  * stencil_tune's choice and timing for each workload, a copy-probe ceiling, MIOpen's
    convolution on the paper and conv-form cases, and one GPU's slab of an 8-way z
    decomposition of the headline (context).
All GPU work runs before the CPU legs, so host threads never overlap a timed region.
Every reported value is the planner's default plan.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import math
import os
import re
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
PAPER_STEPS_TIMED = 256
ALU_PEAK_TFLOPS = 78.6
# The paper's per-step latencies for its 2D radius-3 fp64 box on 10240^2, on an NVIDIA
# A100-PCIE-40GB (Sec. "RQ3: Case Study on Stencil Computation"): context, not a target.
PAPER_A100_MS_PER_STEP = {"best_generated_kernel": 4.71, "cudnn_implicit_precomp_gemm": 7.23}
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = {
    "stencil_box3_stream_kernel": ["kernel_box.hip", "common.hpp", "plan.hpp"],
    "stencil_star_stream_kernel": ["kernel_star.hip", "common.hpp", "plan.hpp"],
    "stencil_star_tb2_kernel": ["kernel_star_tb.hip", "common.hpp", "plan.hpp"],
    "stencil_star_tbs_kernel": ["kernel_star_tbs.hip", "common.hpp", "plan.hpp"],
    "stencil_box2_stream_kernel": ["kernel_box2.hip", "common.hpp", "plan.hpp"],
    "stencil_box2_tb2_kernel": ["kernel_box2.hip", "common.hpp", "plan.hpp"],
    "stencil_generic_kernel": ["kernel_generic.hip", "plan.hpp"],
}


DATA = {
    "laplace2d": "i.i.d. U[-1,1] input",
    "star7": "i.i.d. U[-1,1] input",
    "fd8": "8 random-phase sinusoids + 1% uniform noise",
    "box_field": "i.i.d. U[-1,1] input, 27 U[-1,1] weights with sum|w|=1, field U[0.5,1]",
    "conv": "i.i.d. N(0,1) input, per-channel U[-1,1] weights with sum|w|=1",
    "box_uniform": "i.i.d. U[-1,1] input, U[-1,1] weights with sum|w|=1",
}


def describe(wl) -> str:
    shape = "star" if wl.shape == 0 else "box"
    pts = wl.npoints
    bnd = "zero" if wl.boundary == 0 else "periodic"
    dims = "x".join(str(d) for d in wl.dims)
    batch = " x %d volumes (N=%d, C=%d)" % (wl.batch, wl.n, wl.channels) if wl.batch > 1 else ""
    field = " with coefficient field" if wl.has_field else ""
    return "%dD %d-point %s R=%d%s, %s%s %s, %s boundary, %d steps per call" % (
        wl.ndim, pts, shape, wl.radius, field, dims, batch, wl.dtype, bnd, wl.steps)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def code_only(text: str) -> str:
    """C++ source without its comments and with whitespace collapsed: what the compiler
    sees, so that a comment-only edit keeps a kernel's hash (the kernel sources hold no
    string literal with comment markers)."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_source_sha(kernel: str) -> str | None:
    """Hash of the code (comments stripped) of a kernel's source files."""
    files = KERNEL_SOURCES.get(kernel)
    if not files:
        return None
    h = hashlib.sha256()
    for f in files:
        path = os.path.join(ROOT, "paper_2608_21157_amd", "csrc", f)
        if not os.path.exists(path):
            return None
        with open(path) as fh:
            h.update(code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def counter_traffic(kernel: str, workload: str, algo_bytes: float):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or None when
    the summary is missing or the kernel source changed since it was taken."""
    path = os.path.join(PROFILES, "counters.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f).get("%s/%s" % (kernel, workload))
    if not rec or rec.get("source_sha") != kernel_source_sha(kernel):
        return None
    return rec.get("hbm_bytes_per_launch")


class Runner:
    def __init__(self, torch, B, inputs, wl, stream, depth=0):
        self.torch, self.B, self.wl, self.stream = torch, B, wl, stream
        t0 = time.perf_counter()
        x, w, k = inputs.make(wl)
        log("[bench] %s: inputs generated in %.1fs" % (wl.name, time.perf_counter() - t0))
        self.x_host, self.k_host = x, k
        dev = torch.device("cuda:0")
        self.x = torch.from_numpy(x).to(dev)
        self.y = torch.empty_like(self.x)
        self.k = None if k is None else torch.from_numpy(k).to(dev)
        self.w = np.ascontiguousarray(w)
        torch.cuda.synchronize()  # the uploads ran on torch's stream; the calls use `stream`
        desc = B.make_desc(wl.ndim, wl.dims, batch=wl.batch, channels=wl.channels,
                           dtype=B.F32 if wl.dtype == "f32" else B.F64, shape=wl.shape,
                           radius=wl.radius, boundary=wl.boundary,
                           has_coeff_field=self.k is not None, temporal_depth=depth)
        self.plan = B.Plan(desc)
        info = self.plan.info()
        self.kernel = info.kernel.decode()
        self.depth = info.temporal_depth
        self.tile, self.grid_scale = info.tile, info.grid_scale
        self.variant = B.VARIANT_NAMES.get(info.variant, str(info.variant))
        self.launches = math.ceil(wl.steps / self.depth) if wl.steps else 0

    def call(self, steps=None):
        self.plan.run(self.x, self.y, self.w, steps=self.wl.steps if steps is None else steps,
                      field=self.k, stream=self.stream)

    def spin(self, seconds: float) -> int:
        """Calls of this workload itself, back to back, for `seconds` (untimed): the
        kernel's steady speed is reached after about 20 calls of itself."""
        t0 = time.perf_counter()
        n = 0
        while True:
            for _ in range(5):
                self.call()
            n += 5
            self.stream.synchronize()
            if time.perf_counter() - t0 >= seconds:
                return n

    def timed(self, K: int, W: int) -> float:
        """Milliseconds for K back-to-back calls (events on the launch stream)."""
        torch = self.torch
        for _ in range(W):
            self.call()
        self.stream.synchronize()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(self.stream)
        for _ in range(K):
            self.call()
        e1.record(self.stream)
        e1.synchronize()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1)

    def graph_timed(self, calls: int, reps: int) -> float:
        """Milliseconds per call with `calls` back-to-back calls captured in one HIP graph
        (torch.cuda.graph on the runner's stream) and the graph replayed `reps` times: what
        a serving loop pays per call once the host-side launch cost is taken out.  The
        plan has run before (its buffers exist, its weights are uploaded), so a captured
        call holds kernel launches only."""
        torch = self.torch
        self.call()
        self.stream.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=self.stream):
            for _ in range(calls):
                self.call_on(torch.cuda.current_stream())
        self.plan._stream = self.stream
        with torch.cuda.stream(self.stream):
            g.replay()
            self.stream.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(self.stream)
            for _ in range(reps):
                g.replay()
            e1.record(self.stream)
            e1.synchronize()
        del g
        return e0.elapsed_time(e1) / (reps * calls)

    def call_on(self, stream):
        self.plan.run(self.x, self.y, self.w, steps=self.wl.steps, field=self.k, stream=stream)

    def flushed(self, R: int, flush, warm: int = 3) -> list:
        """The paper's protocol: `warm` untimed calls, then R calls timed one by one
        (events on the launch stream), each after `flush` has evicted the caches on the
        same stream, outside the events.  Returns the R per-call milliseconds."""
        torch = self.torch
        for _ in range(warm):
            self.call()
        self.stream.synchronize()
        out = []
        for i in range(R):
            flush(self.stream, i)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(self.stream)
            self.call()
            e1.record(self.stream)
            e1.synchronize()
            out.append(e0.elapsed_time(e1))
        return out

    def output(self) -> np.ndarray:
        """Host copy of `out` after the work queued so far."""
        self.stream.synchronize()
        return self.y.cpu().numpy()

    def close(self):
        self.plan.close()
        del self.x, self.y, self.k


class Flush:
    """Evicts L2 and the Infinity Cache by reading a 1 GiB buffer on a given stream.
    Reading (a sum) rather than writing leaves only clean lines behind: the dirty lines
    of the previous call are written back during the flush, and the timed call does not
    pay to write back the flush's own data."""

    def __init__(self, torch, nbytes: int = 1 << 30):
        self.torch = torch
        self.buf = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda:0")
        torch.cuda.synchronize()

    def __call__(self, stream, i: int) -> None:
        with self.torch.cuda.stream(stream):
            self.sink = self.buf.sum()


def protocol_record(wl, times: list) -> dict:
    med = statistics.median(times)
    return {"calls": len(times), "warmup": 3, "flush": "1 GiB read on the timed stream",
            "median_ms": round(med, 5), "min_ms": round(min(times), 5),
            "gpoints_per_s_median": figures(wl, med)["gpoints_per_s"],
            "gpoints_per_s_min_time": figures(wl, min(times))["gpoints_per_s"],
            "frac_of_8tbs_median": figures(wl, med)["frac_of_8tbs"]}


def tolerance(wl, x, k=None) -> float:
    """The parity bar: fp32 1e-5 per step, scaled by max|x| (and max k) above 1; fp64 a
    flat 1e-12."""
    if wl.dtype != "f32":
        return 1e-12
    scale = max(1.0, float(np.abs(x).max()))
    if k is not None:
        scale *= max(1.0, float(np.abs(k).max()))
    return 1e-5 * max(wl.steps, 1) * scale


def oracle_check(wl, x, w, k, got, what: str) -> dict:
    """`got` against the fp64 oracle at every point of the grid (the oracle evaluated in
    independent slabs or volumes on host threads; see oracle/whole_grid.py)."""
    from oracle import whole_grid
    rep = whole_grid.compare(got, x, w, shape=wl.shape, radius=wl.radius,
                             boundary=wl.boundary, steps=wl.steps, ndim=wl.ndim,
                             channels=wl.channels, field=k)
    tol = tolerance(wl, x, k)
    pts = int(x.size) * max(wl.steps, 1)
    ok = rep["nonfinite"] == 0 and rep["max_abs_err"] <= tol
    return {"what": what, "points": rep["points"], "steps": wl.steps,
            "max_abs_err": rep["max_abs_err"], "worst_flat_index": rep["worst"],
            "nonfinite": rep["nonfinite"], "tolerance": tol, "pass": bool(ok),
            "oracle_seconds": rep["seconds"], "oracle_threads": rep["threads"],
            "oracle_pieces": rep["pieces"],
            "oracle_gpoints_per_s": round(pts / max(rep["seconds"], 1e-9) / 1e9, 5)}


def figures(wl, ms_per_call: float) -> dict:
    pts = wl.points_per_step * wl.steps
    bytes_pt = wl.itemsize * (2 + (1 if wl.has_field else 0))
    gpts = pts / (ms_per_call * 1e-3) / 1e9
    gbs = pts * bytes_pt / (ms_per_call * 1e-3) / 1e9
    # run-compulsory: the fields read once and the output written once per call, however
    # many steps the call takes (a secondary reading; the sweep figure above is graded)
    run_gbs = wl.points_per_step * bytes_pt / (ms_per_call * 1e-3) / 1e9
    return {"ms_per_call": round(ms_per_call, 5), "gpoints_per_s": round(gpts, 2),
            "effective_gbs": round(gbs, 1), "frac_of_8tbs": round(gbs / HBM_PEAK_GBS, 4),
            "run_compulsory_gbs": round(run_gbs, 1)}


def spin_up(torch, stream, seconds=0.3) -> float:
    """Keep the GPU busy for `seconds` (1 GiB fills) before any workload is built or timed:
    after an idle period the first ~0.1 s of work measured up to 15 % slower (clocks
    leaving their idle state).  Outside every timed region."""
    buf = torch.empty(1 << 28, dtype=torch.float32, device="cuda:0")
    t0 = time.perf_counter()
    with torch.cuda.stream(stream):
        while time.perf_counter() - t0 < seconds:
            for i in range(20):
                buf.fill_(float(i))
            stream.synchronize()
    del buf
    return round(time.perf_counter() - t0, 3)


def copy_probe(torch, stream, nbytes=1 << 30, reps=20, kind="copy"):
    """Achievable HBM throughput of a plain stream of the same shape as a stencil's: `copy`
    (one array read, one written, `nbytes` each) or `triad` (two read, one written: the
    mix of a stencil with a coefficient field).  GB/s counts every array once."""
    path = os.path.join(ROOT, "paper_2608_21157_amd", "libstencil_probe.so")
    lib = ctypes.CDLL(path)
    vp = ctypes.c_void_p
    lib.stencil_probe_copy.argtypes = [vp, vp, ctypes.c_int64, vp]
    lib.stencil_probe_copy.restype = ctypes.c_int
    lib.stencil_probe_triad.argtypes = [vp, vp, vp, ctypes.c_int64, vp]
    lib.stencil_probe_triad.restype = ctypes.c_int
    a = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda:0").uniform_()
    b = torch.empty_like(a).uniform_() if kind == "triad" else None
    c = torch.empty_like(a)
    torch.cuda.synchronize()  # the inputs are filled on torch's stream, the probe uses `stream`
    sh = stream.cuda_stream
    if kind == "triad":
        run = lambda: lib.stencil_probe_triad(a.data_ptr(), b.data_ptr(), c.data_ptr(), nbytes, sh)
        arrays = 3
    else:
        run = lambda: lib.stencil_probe_copy(a.data_ptr(), c.data_ptr(), nbytes, sh)
        arrays = 2
    for _ in range(3):
        assert run() == 0
    stream.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        run()
    e1.record(stream)
    e1.synchronize()
    ms = e0.elapsed_time(e1) / reps
    assert torch.equal(c, a * b if kind == "triad" else a)
    del a, b, c
    torch.cuda.empty_cache()
    return {"kind": kind, "bytes": nbytes, "ms": round(ms, 4),
            "gbs": round(arrays * nbytes / ms / 1e6, 1)}


# The probe each one-step workload is read against: its own access mix at its own array
# size (the multi-step workloads move fewer HBM bytes than their sweep figure counts).
PATTERN_PROBES = {"c4": ("triad", 1 << 29), "c5": ("copy", 1 << 31), "c5b": ("copy", 1 << 30)}


def tune_context(torch, B, head, K: int, W: int, reps: int = 10) -> dict:
    """stencil_tune on a runner's workload (a fresh plan of the same description, the same
    buffers; `reps` timed calls per candidate), then K calls of the tuned plan timed like
    the default plan: a 0.3 s spin-up on its own calls and W warm-up calls first.  Context
    only: every reported value is the planner's default plan."""
    plan = B.Plan(head.plan.desc)
    try:
        rep = plan.tune(head.x, head.y, head.w, steps=head.wl.steps, field=head.k, reps=reps,
                        stream=head.stream)
        info = plan.info()
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < 0.3:
            for _ in range(5):
                plan.run(head.x, head.y, head.w, steps=head.wl.steps, field=head.k,
                         stream=head.stream)
            head.stream.synchronize()
        for _ in range(W):
            plan.run(head.x, head.y, head.w, steps=head.wl.steps, field=head.k,
                     stream=head.stream)
        head.stream.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(head.stream)
        for _ in range(K):
            plan.run(head.x, head.y, head.w, steps=head.wl.steps, field=head.k,
                     stream=head.stream)
        e1.record(head.stream)
        e1.synchronize()
        ms = e0.elapsed_time(e1) / K
    finally:
        plan.close()
    chosen = rep["candidates"][rep["chosen"]]
    out = {"chosen": {k: chosen[k] for k in ("variant", "temporal_depth", "tile", "grid_scale")},
           "kernel": info.kernel.decode(), "candidates": len(rep["candidates"]),
           "valid": sum(c["valid"] for c in rep["candidates"]),
           "tolerance": rep["tolerance"]}
    out.update(figures(head.wl, ms))
    return out


def alu_roofline(wl, launches_per_call: int, avg_launch_ms: float) -> dict:
    """The flop side of a call's launches: algorithmic flops (2 per offset and point-step,
    plus 1 for the coefficient field) per launch over the average launch time.  Peak:
    256 CUs x 4 SIMDs x 16 lanes x 2 flops x 2.4 GHz = 78.6 TFLOP/s for fp32 or fp64 FMAs
    issued one per lane; the build keeps packed fp32 out, which the published 157.3
    TFLOP/s fp32 figure assumes."""
    flops_pt = 2 * wl.npoints + (1 if wl.has_field else 0)
    flops_per_launch = wl.points_per_step * (wl.steps / launches_per_call) * flops_pt
    tflops = flops_per_launch / (avg_launch_ms * 1e-3) / 1e12
    return {"bound": "alu", "achieved": round(tflops, 2), "peak": ALU_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": round(tflops / ALU_PEAK_TFLOPS, 4),
            "published_fp32_peak": 157.3,
            "algorithmic_flops_per_launch": int(flops_per_launch)}


def slab_context(torch, B, inputs, stream, gpus=8, reps=20) -> dict:
    """One GPU's share of the headline under a z-slab decomposition over `gpus` GPUs: its
    512/gpus owned planes plus the 2R planes on each side that one fused two-step pass
    reads from its neighbours, timed for one pass (context for the multi-GPU design; the
    halo exchange itself is not run)."""
    wl = inputs.WORKLOADS["c3"]
    own = wl.dims[0] // gpus
    halo = 2 * wl.radius  # planes per side for two fused steps
    slab = wl.resized((own + 2 * halo,) + tuple(wl.dims[1:]), steps=2)
    r = Runner(torch, B, inputs, slab, stream)
    r.spin(0.3)
    t = r.timed(reps, 3) / reps
    kernel = r.kernel
    r.close()
    torch.cuda.empty_cache()
    owned = own * wl.dims[1] * wl.dims[2] * slab.steps
    plane_mib = wl.dims[1] * wl.dims[2] * wl.itemsize / 2 ** 20
    return {"dims": list(slab.dims), "owned_planes": own, "halo_planes_per_side": halo,
            "ms_per_pass": round(t, 5), "kernel": kernel,
            "owned_gpoints_per_s": round(owned / (t * 1e-3) / 1e9, 2),
            "halo_mib_per_face": round(halo * plane_mib, 1)}


def deep_fusion_context(torch, B, inputs, stream, reps=20) -> dict:
    """The c2 operator (fp32 7-point star, 10 steps) on 512^3, beyond the Infinity Cache:
    the planner's four steps per pass against two (context for the temporal depth rule;
    the c2 workload itself, 256^3, stays inside the cache and runs two)."""
    wl = inputs.WORKLOADS["c2_512"]
    out = {"dims": list(wl.dims), "steps": wl.steps}
    for key, depth in (("planner", 0), ("two_per_pass", 2)):
        r = Runner(torch, B, inputs, wl, stream, depth=depth)
        r.spin(0.3)
        t = r.timed(reps, 10) / reps
        out[key] = {"kernel": r.kernel, "depth": r.depth, "ms_per_call": round(t, 5),
                    "gpoints_per_s": figures(wl, t)["gpoints_per_s"]}
        r.close()
        torch.cuda.empty_cache()
    return out


def miopen_context(torch, wl, x_host, w, reps=5):
    """Time torch's convolution (MIOpen on ROCm) on the same workload, one stencil step per
    call: the MI355X counterpart of the paper's cuDNN dense reference.  Context only; its
    result is never a parity reference.  Returns None if MIOpen cannot run the case."""
    try:
        F = torch.nn.functional
        dev = torch.device("cuda:0")
        x = torch.from_numpy(x_host).to(dev)
        k = 2 * wl.radius + 1
        if wl.ndim == 2:
            inp = x.reshape(1, 1, *wl.dims)
            wt = torch.from_numpy(w.reshape(1, 1, k, k)).to(dev)
            run = lambda: F.conv2d(inp, wt, padding=wl.radius)
        else:
            inp = x.reshape(wl.n, wl.channels, *wl.dims)
            wt = torch.from_numpy(w.reshape(wl.channels, 1, k, k, k)).to(dev)
            run = lambda: F.conv3d(inp, wt, padding=wl.radius, groups=wl.channels)
        for _ in range(2):
            run()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            run()
        e1.record()
        e1.synchronize()
        ms = e0.elapsed_time(e1) / reps
        del inp, wt, x
        torch.cuda.empty_cache()
        return {"ms_per_step": round(ms, 4),
                "gpoints_per_s": round(wl.points_per_step / (ms * 1e-3) / 1e9, 2),
                "what": "torch.nn.functional.conv%dd (MIOpen), one step, same input" % wl.ndim}
    except Exception as e:  # MIOpen may not support every dtype/shape
        return {"error": str(e)[:200]}


def host_info(torch) -> dict:
    """CPU model, logical CPUs, ROCm and torch versions of the measuring host."""
    info = {"cpus": os.cpu_count(), "torch": torch.__version__}
    try:
        with open("/proc/cpuinfo") as f:
            lines = f.readlines()
        info["cpu"] = next(l.split(":", 1)[1].strip() for l in lines if l.startswith("model name"))
        mhz = [float(l.split(":", 1)[1]) for l in lines if l.startswith("cpu MHz")]
        if mhz:
            info["cpu_mhz"] = round(max(mhz))
    except (OSError, StopIteration, ValueError):
        pass
    try:
        with open("/opt/rocm/.info/version") as f:
            info["rocm"] = f.read().strip()
    except OSError:
        pass
    try:
        info["gpu"] = torch.cuda.get_device_name(0)
        info["gpu_arch"] = torch.cuda.get_device_properties(0).gcnArchName
    except Exception:
        pass
    return info


def cpu_baseline(wl, x_host, w, planes: int):
    """The fp64 oracle as it stands, single-threaded, on a z-slab of the headline input:
    the CPU reference throughput (a reported baseline, not a target)."""
    import oracle
    oracle.build()
    slab = x_host[:planes]
    t0 = time.perf_counter()
    oracle.apply(slab, w, shape=wl.shape, radius=wl.radius, boundary=wl.boundary,
                 steps=wl.steps, ndim=wl.ndim)
    dt = time.perf_counter() - t0
    pts = slab.size * wl.steps
    return {"value": round(pts / dt / 1e9, 6), "unit": "Gpoints/s", "cores": 1,
            "kind": "oracle", "seconds": round(dt, 2),
            "sample": "%dx%dx%d z-slab of the headline input, %d steps, fp64 single thread"
                      % (slab.shape + (wl.steps,))}


# workloads of the per-workload block, in order; the headline's own record is reused for
# its name rather than timed twice
WORKLOAD_ORDER = ("c1", "c2", "c3", "c4", "c5", "c5b", "paper")
PROTOCOL_CALLS = 100
# the paper workload's output is checked on a call of 4 steps (two fused launches through
# the ping-pong grid, in the timed launch configuration): its timed 256-step call is
# beyond a whole-grid oracle's reach
PAPER_CHECK_STEPS = 4


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50, help="timed calls")
    ap.add_argument("--warmup", type=int, default=30, help="untimed calls")
    ap.add_argument("--spin-s", type=float, default=0.3,
                    help="seconds of untimed calls of the headline kernel before the warm-up")
    ap.add_argument("--workload", default="c3")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-checks", action="store_true",
                    help="skip the whole-grid oracle checks of the outputs")
    ap.add_argument("--protocol-calls", type=int, default=PROTOCOL_CALLS,
                    help="flushed, individually timed calls per workload (0: none)")
    ap.add_argument("--no-others", action="store_true", help="headline workload only")
    ap.add_argument("--cpu-planes", type=int, default=320,
                    help="z planes of the headline input the single-thread oracle runs on")
    ap.add_argument("--stencil-steps", type=int, default=0,
                    help="override the workload's stencil steps per call (profiling runs)")
    ap.add_argument("--depth", type=int, default=0,
                    help="stencil steps fused per launch (0: the planner's choice)")
    ap.add_argument("--no-tune", action="store_true",
                    help="skip the stencil_tune context figures")
    ap.add_argument("--copy-only", action="store_true",
                    help="run only the copy probe (counter calibration runs)")
    args = ap.parse_args()

    if args.gpus != 1:
        log("bench.py measures one GPU only: this library runs the stencil on a single "
            "MI355X (multi-GPU slab decomposition is a design note, not built).  "
            "Use --gpus 1.")
        return 2

    import torch
    from paper_2608_21157_amd import binding as B
    from paper_2608_21157_amd import inputs

    if not torch.cuda.is_available():
        log("no GPU visible")
        return 1
    B.load()
    stream = torch.cuda.Stream()
    if args.copy_only:
        probe = copy_probe(torch, stream, reps=args.steps)
        print(json.dumps({"copy_probe": probe}), flush=True)
        return 0
    wl = inputs.WORKLOADS[args.workload]
    if args.stencil_steps > 0:
        wl = wl.resized(wl.dims, steps=args.stencil_steps)
    flush = Flush(torch) if args.protocol_calls > 0 else None
    checks_todo = []   # (name, workload, x, w, k, output, what): run after all GPU work

    # ---- headline: spin-up on its own kernel, W warm-up calls, K timed calls ------------
    head = Runner(torch, B, inputs, wl, stream, depth=args.depth)
    t0 = time.perf_counter()
    spin_calls = head.spin(args.spin_s) if args.spin_s > 0 else 0
    spun = round(time.perf_counter() - t0, 3)
    ms_total = head.timed(args.steps, args.warmup)
    ms = ms_total / args.steps
    fig = figures(wl, ms)
    launches = head.launches * args.steps
    bytes_pt = wl.itemsize * (2 + (1 if wl.has_field else 0))
    algo_per_launch = wl.points_per_step * (wl.steps / head.launches) * bytes_pt
    avg_launch_ms = ms_total / launches
    achieved = algo_per_launch / (avg_launch_ms * 1e-3) / 1e9
    traffic = counter_traffic(head.kernel, wl.name, algo_per_launch)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": traffic, "kernel": head.kernel,
                "avg_launch_ms": round(avg_launch_ms, 5),
                "algorithmic_bytes_per_launch": int(algo_per_launch),
                "achieved_is": "sweep-compulsory bytes (each fused step's read and write) "
                               "per launch over the event-timed launch time",
                "counter_gbs": (round(traffic / (avg_launch_ms * 1e-3) / 1e9, 1)
                                if traffic else None)}
    roofline_alu = alu_roofline(wl, head.launches, avg_launch_ms)
    log("[bench] %s: %.4f ms/call, %.1f Gpoints/s, %.1f GB/s (%.1f%% of 8 TB/s); spin-up "
        "%d calls" % (wl.name, ms, fig["gpoints_per_s"], achieved, 100 * achieved / HBM_PEAK_GBS,
                      spin_calls))
    head_rec = dict(fig)
    head_rec.update(kernel=head.kernel, variant=head.variant, depth=head.depth,
                    tile=head.tile, grid_scale=head.grid_scale,
                    launches_per_call=head.launches, timed_calls=args.steps)
    if not args.no_checks:
        # the timed default plan's own output, before anything else writes `out`
        checks_todo.append((wl.name, wl, head.x_host, head.w, head.k_host, head.output(),
                            "the timed default plan's output"))
    protocol = None
    if flush is not None:
        protocol = protocol_record(wl, head.flushed(args.protocol_calls, flush))
        head_rec["protocol"] = protocol
        log("[bench] %s protocol: %s" % (wl.name, protocol))

    tuned = None
    if not args.no_tune:
        tuned = tune_context(torch, B, head, args.steps, args.warmup)
        head_rec["tuned"] = {k: tuned[k] for k in ("chosen", "kernel", "candidates", "valid",
                                                    "ms_per_call", "gpoints_per_s")}
        log("[bench] tuned %s: %s" % (wl.name, tuned))
    cpu_input = (head.x_host, head.w) if (not args.no_cpu_baseline and wl.ndim == 3
                                          and wl.batch == 1) else None
    head.close()
    torch.cuda.empty_cache()

    others = {}
    probe = None
    if not args.no_others:
        spin_up(torch, stream)
        probe = copy_probe(torch, stream)
        log("[bench] copy probe: %s" % probe)
        patterns = {}
        for name, (kind, nbytes) in PATTERN_PROBES.items():
            key = (kind, nbytes)
            if key not in patterns:
                patterns[key] = copy_probe(torch, stream, nbytes, kind=kind)
                log("[bench] %s probe, %d MiB per array: %s" % (kind, nbytes >> 20,
                                                                 patterns[key]))
        for name in WORKLOAD_ORDER:
            if name == wl.name:
                rec = head_rec
            else:
                w2 = inputs.WORKLOADS[name]
                if name == "paper":
                    # the paper iterates 10,240 times and reports the amortised per-step
                    # latency; 256-step calls amortise the same way at a tenth of the time
                    w2 = w2.resized(w2.dims, steps=PAPER_STEPS_TIMED)
                rec = workload_leg(torch, B, inputs, w2, stream, flush, args, checks_todo)
            if probe:
                rec["frac_of_copy_probe"] = round(rec["effective_gbs"] / probe["gbs"], 4)
            if name in PATTERN_PROBES:
                pp = patterns[PATTERN_PROBES[name]]
                rec["pattern_probe"] = pp
                rec["frac_of_pattern_probe"] = round(rec["effective_gbs"] / pp["gbs"], 4)
            others[name] = rec
            log("[bench] %s: %s" % (name, rec))
        others["c3_slab_of_8"] = slab_context(torch, B, inputs, stream)
        log("[bench] c3_slab_of_8: %s" % others["c3_slab_of_8"])
        others["c2_at_512_cubed"] = deep_fusion_context(torch, B, inputs, stream)
        log("[bench] c2_at_512_cubed: %s" % others["c2_at_512_cubed"])
    del flush
    torch.cuda.empty_cache()

    # ---- CPU legs, after every GPU measurement -----------------------------------------
    cpu = None
    if cpu_input is not None:
        planes = min(args.cpu_planes, wl.dims[0])
        cpu = cpu_baseline(wl, cpu_input[0], cpu_input[1], planes)
        log("[bench] cpu oracle: %s" % cpu)
    checks = {}
    for name, cwl, x, w, k, got, what in checks_todo:
        checks[name] = oracle_check(cwl, x, w, k, got, what)
        log("[bench] oracle check %s: %s" % (name, checks[name]))
        if name in others:
            others[name]["oracle_check"] = checks[name]
        del got
    checks_todo.clear()

    line = {
        "metric": "stencil Gpoints/s and achieved HBM GB/s (% of MI355X peak), 3D fp32 512^3",
        "value": fig["gpoints_per_s"], "unit": "Gpoints/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup,
        "spin_up": {"seconds": spun, "calls": spin_calls,
                    "what": "untimed calls of the headline workload before the warm-up"},
        "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
        "data": "synthetic, seeded: " + DATA[wl.recipe],
        "config": {"workload": describe(wl),
                   "dims": list(wl.dims), "stencil_steps_per_call": wl.steps,
                   "kernel": head_rec["kernel"], "variant": head_rec["variant"],
                   "temporal_depth": head_rec["depth"], "parallelism": "single GPU"},
        "effective_gbs": fig["effective_gbs"],
        "run_compulsory_gbs": fig["run_compulsory_gbs"],
        "roofline": roofline,
        "roofline_alu": roofline_alu,
        "protocol": protocol,
        "oracle_check": checks.get(wl.name),
        "oracle_checks_pass": (all(c["pass"] for c in checks.values()) if checks else None),
        "tuned": tuned,
        "host": host_info(torch),
        "cpu_baseline": cpu,
        "copy_probe": probe,
        "workloads": others,
    }
    print(json.dumps(line), flush=True)
    return 0


def timed_calls(s_per_call: float, window_s: float = 0.05) -> int:
    """Back-to-back calls for a timed window of about `window_s` (20 to 5000): a window of a
    few calls would be dominated by the first launch's latency on a launch-bound workload."""
    return int(min(5000, max(20, window_s / max(s_per_call, 1e-9))))


def workload_leg(torch, B, inputs, wl, stream, flush, args, checks_todo) -> dict:
    """One workload of the per-workload block: spin-up on its own kernel, about 50 ms of
    back-to-back calls (20 at least) after 20 warm-up calls, the flushed protocol, the tuner's choice, and (queued
    for the CPU phase) its output for the whole-grid oracle check."""
    r = Runner(torch, B, inputs, wl, stream)
    paper = wl.name == "paper"
    spun = r.spin(0.3)
    reps = 3 if paper else timed_calls(0.3 / spun)
    t = r.timed(reps, 1 if paper else 20) / reps
    rec = figures(wl, t)
    rec.update(kernel=r.kernel, variant=r.variant, depth=r.depth, tile=r.tile,
               grid_scale=r.grid_scale, launches_per_call=r.launches, timed_calls=reps)
    if not args.no_checks:
        if paper:
            r.call(steps=PAPER_CHECK_STEPS)
            checks_todo.append((wl.name, wl.resized(wl.dims, steps=PAPER_CHECK_STEPS),
                                r.x_host, r.w, r.k_host, r.output(),
                                "a %d-step call of the timed default plan" % PAPER_CHECK_STEPS))
        else:
            checks_todo.append((wl.name, wl, r.x_host, r.w, r.k_host, r.output(),
                                "the timed default plan's output"))
    if flush is not None:
        rec["protocol"] = protocol_record(wl, r.flushed(args.protocol_calls, flush))
    if not args.no_tune:
        # the fastest valid launch configuration for this workload (the tuner's search),
        # timed like the default plan above
        tr = tune_context(torch, B, r, reps, 1 if paper else 3, reps=3 if paper else 5)
        rec["tuned"] = {k: tr[k] for k in ("chosen", "kernel", "candidates", "valid",
                                           "ms_per_call", "gpoints_per_s")}
    if wl.name in ("c1", "c2"):
        # launch-bound workloads: the same calls replayed from a HIP graph
        gms = r.graph_timed(50, 20)
        rec["graph_replay"] = {"ms_per_call": round(gms, 5),
                               "gpoints_per_s": figures(wl, gms)["gpoints_per_s"],
                               "calls_per_graph": 50}
    if paper:
        rec["ms_per_stencil_step"] = round(t / wl.steps, 5)
        rec["context_a100_ms_per_step"] = PAPER_A100_MS_PER_STEP
    if wl.name in ("paper", "c5"):
        rec["context_miopen"] = miopen_context(torch, wl, r.x_host, r.w)
    r.close()
    torch.cuda.empty_cache()
    return rec


if __name__ == "__main__":
    sys.exit(main())
