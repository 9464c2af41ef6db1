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
