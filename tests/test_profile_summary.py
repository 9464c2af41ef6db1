"""The profiler wrapper's summary step on synthetic rocprofv3 outputs (no GPU): counter
calibration against the copy probe, traffic per launch, and the counters.json record that
bench.py reads for its roofline ``traffic`` figure."""
import csv
import json
import os

from paper_2608_21157_amd import profile

import bench


def _write_csv(path, header, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


STATS = ["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs", "MaxNs",
         "StdDev"]
PMC = ["Kernel_Name", "Counter_Name", "Counter_Value"]


def _fake_run(out, kernel, workload, avg_ns, fetch_kib, write_kib):
    _write_csv(os.path.join(out, "trace_" + workload, workload + "_kernel_stats.csv"), STATS,
               [["void fill_kernel<float>(...)", 100, 1000, 10, 1.0, 9, 11, 0],
                ["void stencil::%s<float, 1>(...)" % kernel, 4, 4 * avg_ns, avg_ns, 99.0,
                 avg_ns, avg_ns, 0]])
    for c, v in (("FETCH_SIZE", fetch_kib), ("WRITE_SIZE", write_kib)):
        _write_csv(os.path.join(out, "pmc_%s_%s" % (c, workload),
                                workload + "_counter_collection.csv"), PMC,
                   [["void stencil::%s<float, 1>(...)" % kernel, c, v]] * 2)


def test_summaries_calibrate_counters_and_record_traffic(tmp_path):
    out, dest = str(tmp_path / "raw"), str(tmp_path / "profiles")
    gib_kib = (1 << 30) // 1024
    # copy probe: FETCH_SIZE reads half the true bytes, WRITE_SIZE all of them
    _fake_run(out, "stencil_probe_copy_kernel", "copy", 370000, gib_kib / 2, gib_kib)
    # c2: the fused star kernel, 2 steps per launch over 256^3 fp32 points
    n = 256 ** 3
    _fake_run(out, "stencil_star_tb2_kernel", "c2", 26000, n * 4 / 1024 / 2 / 2, n * 4 / 1024)
    # one pass ended with a non-zero status after writing its results
    for name, _, _, _ in profile.passes("c2") + profile.passes("copy"):
        profile.record_status(out, name, {"status": 139 if name == "pmc_SQ_c2" else 0,
                                          "seconds": 3.0, "complete": True})
    rec = profile.write_summaries(out, ["c2"], dest=dest)["stencil_star_tb2_kernel/c2"]
    assert rec["fetch_scale"] == 2.0 and rec["write_scale"] == 1.0
    assert rec["algorithmic_bytes_per_launch"] == 8 * n * 2
    assert rec["hbm_bytes_per_launch"] == n * 4 // 2 + n * 4    # half the input, all outputs
    assert abs(rec["traffic_over_algorithmic"] - 0.375) < 1e-9
    assert rec["source_sha"] == bench.kernel_source_sha("stencil_star_tb2_kernel")
    with open(os.path.join(dest, "counters.json")) as f:
        assert json.load(f) == {"stencil_star_tb2_kernel/c2": rec}
    text = open(os.path.join(dest, "star_tb2_c2_256x256x256_f32.txt")).read()
    assert "rocprofv3 --pmc FETCH_SIZE" in text and "--workload c2" in text
    assert "0.375 x algorithmic" in text
    assert "pmc_FETCH_SIZE_c2 0 (3 s)" in text and "pmc_SQ_c2 139 (3 s)" in text
    assert "non-zero exit kept for their complete results: pmc_SQ_c2" in text
    assert os.path.exists(os.path.join(dest, "copy_probe_1GiB_calibration.txt"))


def test_pass_list_uses_one_counter_group_per_pass():
    for w in profile.WORKLOADS + ("copy",):
        for name, opts, args, limit in profile.passes(w):
            if "--pmc" in opts:
                counters = opts[opts.index("--pmc") + 1:]
                sq = [c for c in counters if c.startswith("SQ_")]
                assert len(sq) <= 8 and (len(counters) == 1 or len(sq) == len(counters))
            assert "--sys-trace" not in opts and "--runtime-trace" not in opts
            assert 0 < limit <= 300
