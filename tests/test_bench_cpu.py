"""bench.py host logic on the CPU: the single-GPU contract, the metric arithmetic and the
source-hash gate on the committed counter records."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2608_21157_amd.inputs import WORKLOADS  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr + r.stdout
    assert r.stdout.strip() == ""  # no JSON line


def test_figures_of_the_headline_workload():
    wl = WORKLOADS["c3"]                      # 512^3 f32, 4 steps per call
    f = bench.figures(wl, 0.5)                # 0.5 ms per call
    pts = 512 ** 3 * 4
    assert f["gpoints_per_s"] == pytest.approx(pts / 0.5e-3 / 1e9, rel=1e-4)
    assert f["effective_gbs"] == pytest.approx(pts * 8 / 0.5e-3 / 1e9, rel=1e-4)
    assert f["frac_of_8tbs"] == pytest.approx(f["effective_gbs"] / 8000, abs=1e-4)
    # read once and written once per call: a quarter of the four-step sweep figure
    assert f["run_compulsory_gbs"] == pytest.approx(f["effective_gbs"] / 4, rel=1e-3)


def test_figures_count_the_coefficient_field():
    wl = WORKLOADS["c4"]                      # in + field + out, f32, one step
    f = bench.figures(wl, 1.0)
    assert f["effective_gbs"] == pytest.approx(512 ** 3 * 12 / 1e-3 / 1e9, rel=1e-4)
    assert f["run_compulsory_gbs"] == pytest.approx(f["effective_gbs"], rel=1e-3)


def test_counter_traffic_only_for_the_profiled_sources():
    path = os.path.join(ROOT, "profiles", "counters.json")
    records = json.load(open(path))
    assert records
    for key, rec in records.items():
        kernel, workload = key.split("/")
        got = bench.counter_traffic(kernel, workload, rec["algorithmic_bytes_per_launch"])
        if rec["source_sha"] == bench.kernel_source_sha(kernel):
            assert got == rec["hbm_bytes_per_launch"]
        else:
            assert got is None
    assert bench.counter_traffic("no_such_kernel", "c3", 1.0) is None


def test_alu_roofline_of_the_fused_headline():
    wl = WORKLOADS["c3"]                      # 25-point star, two launches of two steps
    r = bench.alu_roofline(wl, 2, 0.336)
    flops = 512 ** 3 * 2 * 50                 # points x fused steps x 2 flops per offset
    assert r["algorithmic_flops_per_launch"] == flops
    assert r["achieved"] == pytest.approx(flops / 0.336e-3 / 1e12, abs=0.01)
    assert r["peak"] == pytest.approx(256 * 4 * 16 * 2 * 2.4e9 / 1e12, abs=0.05)
    assert r["frac"] == pytest.approx(r["achieved"] / r["peak"], abs=1e-3)


def test_alu_roofline_counts_the_field_multiply():
    wl = WORKLOADS["c4"]                      # 27-point box with k[p], one step
    r = bench.alu_roofline(wl, 1, 1.0)
    assert r["algorithmic_flops_per_launch"] == 512 ** 3 * (2 * 27 + 1)


def test_code_hash_ignores_comments_but_not_code():
    src = "int f(int a) {  // one\n  /* two\n lines */ return a + 1;\n}\n"
    same = "int f(int a) { return a + 1; }  // other comment\n"
    other = "int f(int a) { return a + 2; }\n"
    assert bench.code_only(src) == bench.code_only(same)
    assert bench.code_only(src) != bench.code_only(other)


def test_tolerance_rule():
    import numpy as np
    x = np.full(8, 0.5, np.float32)
    assert bench.tolerance(WORKLOADS["c3"], x) == pytest.approx(4e-5)          # 1e-5 x 4 steps
    big = np.array([-6.0, 2.0], np.float32)
    assert bench.tolerance(WORKLOADS["c5"], big) == pytest.approx(6e-5)        # x max|x|
    k = np.array([0.5, 2.0], np.float32)
    assert bench.tolerance(WORKLOADS["c4"], x, k) == pytest.approx(2e-5)       # x max k
    assert bench.tolerance(WORKLOADS["c5b"], big * 100) == 1e-12               # flat fp64
    assert bench.tolerance(WORKLOADS["paper"], x) == 1e-12


def test_protocol_record_grades_the_median():
    wl = WORKLOADS["c3"]
    rec = bench.protocol_record(wl, [0.7, 0.5, 0.6, 0.9])
    assert rec["median_ms"] == pytest.approx(0.65) and rec["min_ms"] == 0.5
    assert rec["gpoints_per_s_median"] == bench.figures(wl, 0.65)["gpoints_per_s"]
    assert rec["calls"] == 4


@pytest.mark.parametrize("name,dims", [("c3", (13, 11, 16)), ("c4", (9, 7, 8)),
                                       ("c5b", (5, 6, 8)), ("paper", (20, 17))])
def test_oracle_check_passes_the_oracle_and_fails_a_planted_error(name, dims):
    """The bench's whole-grid check accepts the oracle's own result rounded to the
    workload's dtype, and flags one perturbed point (and a NaN)."""
    import numpy as np
    import oracle
    from paper_2608_21157_amd import inputs
    wl = WORKLOADS[name].resized(dims, n=1 if WORKLOADS[name].batch > 1 else None,
                                 steps=min(WORKLOADS[name].steps, 3))
    x, w, k = inputs.make(wl)
    ref = oracle.apply(x, w, shape=wl.shape, radius=wl.radius, boundary=wl.boundary,
                       steps=wl.steps, field=k, ndim=wl.ndim, channels=wl.channels)
    got = ref.astype(x.dtype)
    rec = bench.oracle_check(wl, x, w, k, got, "test")
    assert rec["pass"] and rec["points"] == x.size and rec["nonfinite"] == 0
    bad = got.copy()
    bad.flat[x.size // 2] += 10 * rec["tolerance"]
    rec = bench.oracle_check(wl, x, w, k, bad, "test")
    assert not rec["pass"] and rec["worst_flat_index"] == x.size // 2
    bad.flat[0] = np.nan
    rec = bench.oracle_check(wl, x, w, k, bad, "test")
    assert not rec["pass"] and rec["nonfinite"] == 1


def test_timed_window_of_the_per_workload_legs():
    assert bench.timed_calls(3.5e-6) == 5000        # launch-bound: capped
    assert bench.timed_calls(0.125e-3) == 400       # about 50 ms
    assert bench.timed_calls(0.63e-3) == 79
    assert bench.timed_calls(10e-3) == 20           # at least 20
    assert bench.timed_calls(0.0) == 5000
