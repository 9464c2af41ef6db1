"""rocprofv3 passes over ``bench.py`` and their summaries (``profiles/*.txt``,
``profiles/counters.json``).

    python -m paper_2608_21157_amd.profile --out OUT [--workloads c3 c4 ...] [--write]

For each workload, five passes profile the bench's headline leg:
  * a kernel-trace pass (``--kernel-trace --stats``), timed like the bench (30 warm-up and
    50 timed calls; the paper workload with 64-step calls);
  * two counter passes, FETCH_SIZE and then WRITE_SIZE (HBM-side bytes);
  * an SQ pass: waves, busy and wave cycles, VALU and LDS instruction counts and activity,
    and LDS bank-conflict cycles;
  * an SQ stall pass: wave cycles spent waiting (any, instruction dependencies, LDS) and
    issuing (any, LDS, scalar), and scalar instruction counts.
The copy probe is traced and counted the same way; its known byte counts calibrate
FETCH_SIZE and WRITE_SIZE.  On gfx950, FETCH_SIZE counts 128-byte requests at half their
size, which the copy calibration shows as a factor of 2.

Each counter pass asks for one counter group only: rocprofv3 does not split counters
over passes, and one request beyond a block's counter slots stalls it.  Every pass runs
under a hard time limit (SIGKILL), from /tmp with TMPDIR=/tmp, with the program itself
after ``--``.  Every pass's exit status and wall time are written to
``OUT/pass_status.json`` and repeated in each summary.  A pass that ends with a non-zero
status after writing complete results is kept, and its status is recorded beside its
figures (rocprofv3 can fault in its own teardown after the program has finished); a
pass killed at its limit, or one that left no results, stops the run.  The counter
passes run the bench with few calls (one warm-up and one timed call, no spin-up): each
counter-collected dispatch is serialised, so a pass over thousands of dispatches (the
paper workload's 10,240-step calls once were) does not finish in its limit.

``--write`` turns the raw outputs in OUT into the summaries under ``profiles/``: one
text file per kernel and workload, giving the commands, the kernel statistics and the
derived traffic, and ``counters.json`` (records of the summarised workloads are
replaced, others kept), which ``bench.py`` reads for the ``traffic`` figure of its
roofline object.  Each record carries the hash of the kernel's sources, so
a record taken from older sources is ignored.
"""
from __future__ import annotations

import argparse
import csv
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")
PROFILES = os.path.join(ROOT, "profiles")
sys.path.insert(0, ROOT)

WORKLOADS = ("c3", "c4", "c2", "c5", "c5b", "paper", "c1", "c2_512")
KERNELS = {  # kernel base name -> short name of the summary file
    "stencil_star_stream_kernel": "star_stream",
    "stencil_star_tb2_kernel": "star_tb2",
    "stencil_star_tbs_kernel": "star_tbs",
    "stencil_box3_stream_kernel": "box3_stream",
    "stencil_box2_stream_kernel": "box2_stream",
    "stencil_box2_tb2_kernel": "box2_tb2",
}
COPY_KERNEL = "stencil_probe_copy_kernel"
COPY_BYTES = 1 << 30
SQ_COUNTERS = ("SQ_WAVES", "SQ_WAVE_CYCLES", "SQ_BUSY_CYCLES", "SQ_INSTS_VALU",
               "SQ_ACTIVE_INST_VALU", "SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT",
               "SQ_LDS_IDX_ACTIVE")
# where the wave cycles go: waiting (for anything, for an instruction's dependencies, for
# LDS results) and issuing (any instruction, LDS, scalar), all in the units of
# SQ_WAVE_CYCLES; one pass (8 SQ counters)
SQ_STALL_COUNTERS = ("SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_WAIT_INST_LDS", "SQ_ACTIVE_INST_ANY",
                     "SQ_ACTIVE_INST_LDS", "SQ_ACTIVE_INST_SCA", "SQ_INSTS_SALU",
                     "SQ_INSTS_SMEM")
PAPER_STEPS = 64  # stencil steps per call of the paper workload under the profiler
# SQ_WAVE_CYCLES counts wave residency in units of 4 cycles and SQ_BUSY_CYCLES sums the
# busy cycles of the shader engines (8 CUs each on MI355X), so the mean resident waves
# per CU is 4 * WAVE_CYCLES / BUSY_CYCLES / 8.  Check: the fused star kernel on c3 keeps
# exactly 11 waves per CU for its whole run, and this gives 10.9.
CUS_PER_SE = 8


def occupancy(wave_cycles: float, busy_cycles: float) -> float:
    return 4.0 * wave_cycles / busy_cycles / CUS_PER_SE


def bench_args(workload: str, timed: bool) -> list:
    """bench.py arguments of one pass: the headline leg only, no tuner, no CPU leg, no
    oracle check and no flushed protocol; the counter passes without the spin-up."""
    args = ["--no-others", "--no-cpu-baseline", "--no-tune", "--no-checks",
            "--protocol-calls", "0", "--workload", workload]
    if not timed:
        args += ["--spin-s", "0"]
    if workload == "paper":
        args += ["--stencil-steps", str(PAPER_STEPS)]
        args += ["--steps", "3", "--warmup", "1"] if timed else ["--steps", "1", "--warmup", "1"]
    else:
        args += ["--steps", "50", "--warmup", "30"] if timed else ["--steps", "1", "--warmup", "1"]
    return args


def passes(workload: str) -> list:
    """(directory name, rocprofv3 options, bench arguments, time limit in s) per pass."""
    if workload == "copy":
        return [("trace_copy", ["--kernel-trace", "--stats"], ["--copy-only", "--steps", "20"], 300),
                ("pmc_FETCH_SIZE_copy", ["--pmc", "FETCH_SIZE"], ["--copy-only", "--steps", "3"], 120),
                ("pmc_WRITE_SIZE_copy", ["--pmc", "WRITE_SIZE"], ["--copy-only", "--steps", "3"], 120)]
    return [("trace_" + workload, ["--kernel-trace", "--stats"], bench_args(workload, True), 300),
            ("pmc_FETCH_SIZE_" + workload, ["--pmc", "FETCH_SIZE"], bench_args(workload, False), 150),
            ("pmc_WRITE_SIZE_" + workload, ["--pmc", "WRITE_SIZE"], bench_args(workload, False), 150),
            ("pmc_SQ_" + workload, ["--pmc"] + list(SQ_COUNTERS), bench_args(workload, False), 150),
            ("pmc_SQSTALL_" + workload, ["--pmc"] + list(SQ_STALL_COUNTERS),
             bench_args(workload, False), 150)]


def command(opts, name, workload, args, out="OUT", bench="R/bench.py") -> list:
    return (["rocprofv3"] + opts + ["--output-format", "csv", "-d", "%s/%s" % (out, name),
                                    "-o", workload, "--", "python3", bench] + args)


STATUS_FILE = "pass_status.json"


def record_status(out: str, name: str, rec: dict) -> None:
    path = os.path.join(out, STATUS_FILE)
    data = {}
    if os.path.exists(path):
        with open(path) as f:
            data = json.load(f)
    data[name] = rec
    with open(path, "w") as f:
        json.dump(data, f, indent=1)


def run_passes(out: str, workloads) -> None:
    """Run every pass of the workloads (and of the copy probe); stop at the first pass
    killed at its limit or left without results.  Each pass's status is recorded."""
    import time
    env = dict(os.environ, TMPDIR="/tmp")
    for w in list(workloads) + ["copy"]:
        for name, opts, args, limit in passes(w):
            cmd = command(opts, name, w, args, out=os.path.abspath(out), bench=BENCH)
            cmd[cmd.index("python3")] = sys.executable
            print("== %s" % name, flush=True)
            log = open(os.path.join(out, name + ".log"), "w")
            t0 = time.time()
            try:
                r = subprocess.run(cmd, cwd="/tmp", env=env, stdout=log, stderr=subprocess.STDOUT,
                                   timeout=limit)
                status = r.returncode
            except subprocess.TimeoutExpired:
                record_status(out, name, {"status": "killed at the %d s limit" % limit,
                                          "seconds": round(time.time() - t0, 1),
                                          "complete": False})
                raise SystemExit("%s: killed at its %d s limit" % (name, limit))
            finally:
                log.close()
            complete = results_complete(out, name, w)
            record_status(out, name, {"status": status, "seconds": round(time.time() - t0, 1),
                                      "complete": complete})
            print("   exit status %d, results %s" % (status, "complete" if complete else
                                                      "missing"), flush=True)
            if status != 0 and not complete:
                raise SystemExit("%s: rocprofv3 exited with %d (see %s.log)" % (name, status, name))


def results_complete(out: str, name: str, workload: str) -> bool:
    suffix = "kernel_stats.csv" if name.startswith("trace") else "counter_collection.csv"
    return os.path.exists(os.path.join(out, name, "%s_%s" % (workload, suffix)))


# ------------------------------------------------------------------------------ summaries

def kernel_stats(out: str, workload: str) -> list:
    with open(os.path.join(out, "trace_" + workload, workload + "_kernel_stats.csv")) as f:
        return list(csv.DictReader(f))


def counters(out: str, workload: str, group: str, kernel: str) -> dict:
    """Mean value per dispatch of each counter of a pass, over the kernel's dispatches
    (empty when the pass left no results)."""
    path = os.path.join(out, "pmc_%s_%s" % (group, workload), workload + "_counter_collection.csv")
    vals = {}
    if not os.path.exists(path):
        return {}
    with open(path) as f:
        for row in csv.DictReader(f):
            if kernel in row["Kernel_Name"]:
                vals.setdefault(row["Counter_Name"], []).append(float(row["Counter_Value"]))
    return {k: (sum(v) / len(v), len(v)) for k, v in vals.items()}


def steady_durations(out: str, workload: str, kernel: str, last: int = 100):
    """(median, mean of the last `last` launches) of a kernel's durations in ns from the
    trace pass, or None: the summary's plain average also counts the first calls, which
    run slower while the GPU warms up."""
    path = os.path.join(out, "trace_" + workload, workload + "_kernel_trace.csv")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = [int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in csv.DictReader(f)
             if kernel in r["Kernel_Name"]]
    if not d:
        return None
    d_sorted = sorted(d)
    tail = d[-last:]
    return d_sorted[len(d_sorted) // 2], sum(tail) / len(tail), len(tail)


def copy_calibration(out: str) -> tuple:
    fetch = counters(out, "copy", "FETCH_SIZE", COPY_KERNEL)["FETCH_SIZE"][0]
    write = counters(out, "copy", "WRITE_SIZE", COPY_KERNEL)["WRITE_SIZE"][0]
    return COPY_BYTES / (fetch * 1024), COPY_BYTES / (write * 1024), fetch, write


def pass_statuses(out: str) -> dict:
    path = os.path.join(out, STATUS_FILE)
    if not os.path.exists(path):
        return {}
    with open(path) as f:
        return json.load(f)


def fmt_cmds(workload: str, statuses: dict | None = None) -> str:
    lines = ["# commands (run from /tmp with TMPDIR=/tmp; R = repository root; or all of them"
             " through `python -m paper_2608_21157_amd.profile --out OUT --write`):"]
    for name, opts, args, _ in passes(workload):
        lines.append("#   " + " ".join(command(opts, name, workload, args)))
    if statuses is not None:
        parts = []
        for name, _, _, _ in passes(workload):
            st = statuses.get(name)
            parts.append("%s %s" % (name, "not recorded" if st is None else
                                    "%s (%.0f s)" % (st["status"], st.get("seconds", 0))))
        lines.append("# exit status of each pass: " + ", ".join(parts))
        bad = [n for n, _, _, _ in passes(workload)
               if statuses.get(n) and statuses[n]["status"] != 0]
        if bad:
            lines.append("# passes with a non-zero exit kept for their complete results: "
                         + ", ".join(bad))
    return "\n".join(lines) + "\n"


def fused_depth(kernel: str, wl) -> int:
    """Stencil steps per launch of the profiled kernel: 2 for the two-step kernels, the
    planner's depth for the kernel of three or four steps (asked of the library, which
    plans on the host), 1 for the one-step kernels."""
    if "tb2" in kernel:
        return 2
    if "tbs" in kernel:
        from paper_2608_21157_amd import binding as B
        d = B.make_desc(wl.ndim, wl.dims, batch=wl.batch, channels=wl.channels,
                        dtype=B.F32 if wl.dtype == "f32" else B.F64, shape=wl.shape,
                        radius=wl.radius, boundary=wl.boundary, has_coeff_field=wl.has_field)
        h = B.stencil_plan(d)
        try:
            return int(B.stencil_plan_query(h).temporal_depth)
        finally:
            B.stencil_destroy(h)
    return 1


def write_summaries(out: str, workloads, dest: str = PROFILES) -> dict:
    import bench
    from paper_2608_21157_amd.inputs import WORKLOADS as WL

    os.makedirs(dest, exist_ok=True)
    statuses = pass_statuses(out)
    fscale, wscale, cf, cw = copy_calibration(out)
    cst = [r for r in kernel_stats(out, "copy") if COPY_KERNEL in r["Name"]][0]
    with open(os.path.join(dest, "copy_probe_1GiB_calibration.txt"), "w") as f:
        f.write("# Copy probe, 1 GiB read + 1 GiB written per dispatch (counter calibration)\n")
        f.write(fmt_cmds("copy", statuses))
        f.write("kernel                      %s\n" % COPY_KERNEL)
        f.write("calls                       %s\n" % cst["Calls"])
        f.write("average duration (ns)       %.0f\n" % float(cst["AverageNs"]))
        f.write("achieved read+write         %.1f GB/s\n" % (2 * COPY_BYTES / float(cst["AverageNs"])))
        f.write("FETCH_SIZE per dispatch     %.1f KiB   (true read: %d KiB)\n" % (cf, COPY_BYTES // 1024))
        f.write("WRITE_SIZE per dispatch     %.1f KiB   (true write: %d KiB)\n" % (cw, COPY_BYTES // 1024))
        f.write("scale factors               FETCH x%.4f, WRITE x%.4f\n" % (fscale, wscale))
    records = {}
    for w in workloads:
        wl = WL[w]
        if w == "paper":
            wl = wl.resized(wl.dims, steps=PAPER_STEPS)
        stats = kernel_stats(out, w)
        top = sorted([r for r in stats if any(k in r["Name"] for k in KERNELS)],
                     key=lambda r: -float(r["TotalDurationNs"]))[0]
        kern = [k for k in KERNELS if k in top["Name"]][0]
        fetch, nf = counters(out, w, "FETCH_SIZE", kern)["FETCH_SIZE"]
        write, nw = counters(out, w, "WRITE_SIZE", kern)["WRITE_SIZE"]
        sq = counters(out, w, "SQ", kern)
        depth = fused_depth(kern, wl)
        bytes_pt = wl.itemsize * (2 + (1 if wl.has_field else 0))
        algo = wl.points_per_step * depth * bytes_pt
        avg_ns = float(top["AverageNs"])
        hbm = fetch * 1024 * fscale + write * 1024 * wscale
        sha = bench.kernel_source_sha(kern)
        records["%s/%s" % (kern, w)] = {
            "source_sha": sha, "avg_launch_ns": round(avg_ns, 1),
            "fetch_kib_per_dispatch": round(fetch, 1), "write_kib_per_dispatch": round(write, 1),
            "fetch_scale": round(fscale, 4), "write_scale": round(wscale, 4),
            "hbm_bytes_per_launch": int(hbm), "algorithmic_bytes_per_launch": int(algo),
            "steady_launch_ns": round(steady_durations(out, w, kern)[1], 1)
            if steady_durations(out, w, kern) else None,
            "traffic_over_algorithmic": round(hbm / algo, 4)}
        fname = "%s_%s_%s_%s.txt" % (KERNELS[kern], w, "x".join(map(str, wl.dims)), wl.dtype)
        with open(os.path.join(dest, fname), "w") as f:
            f.write("# %s on %s\n" % (kern, bench.describe(wl)))
            f.write(fmt_cmds(w, statuses))
            f.write("# kernel source sha256[:16] of the profiled build: %s\n" % sha)
            f.write("kernel stats (--kernel-trace --stats):\n")
            for r in stats:
                f.write("  %-100s calls %4d  avg %12.1f ns  %6.2f %%\n" % (
                    r["Name"][:100], int(r["Calls"]), float(r["AverageNs"]), float(r["Percentage"])))
            sd = steady_durations(out, w, kern)
            if sd:
                f.write("duration median (ns)              %.1f\n" % sd[0])
                f.write("duration, mean of the last %d     %.1f  (steady state; the average above"
                        " also counts the warm-up launches)\n" % (sd[2], sd[1]))
            f.write("stencil steps per launch          %d\n" % depth)
            f.write("algorithmic bytes per launch      %d  (%d B per point-step x %d points x %d)\n"
                    % (algo, bytes_pt, wl.points_per_step, depth))
            f.write("achieved (algorithmic / avg)      %.1f GB/s  = %.4f of 8 TB/s\n"
                    % (algo / avg_ns, algo / avg_ns / 8000))
            if sd:
                f.write("achieved (algorithmic / steady)   %.1f GB/s  = %.4f of 8 TB/s\n"
                        % (algo / sd[1], algo / sd[1] / 8000))
            f.write("FETCH_SIZE per dispatch           %.1f KiB  (n=%d) x %.4f (copy calibration)\n"
                    % (fetch, nf, fscale))
            f.write("WRITE_SIZE per dispatch           %.1f KiB  (n=%d) x %.4f\n" % (write, nw, wscale))
            f.write("HBM-side traffic per launch       %d B = %.3f x algorithmic\n" % (int(hbm), hbm / algo))
            if sq:
                f.write("SQ counters per dispatch (sums over the sampled shader engines):\n")
            for c in SQ_COUNTERS:
                if c in sq:
                    f.write("  %-24s %16.0f\n" % (c, sq[c][0]))
            if sq.get("SQ_LDS_IDX_ACTIVE", (0,))[0] > 0:
                f.write("  LDS cycles stalled on bank conflicts: %.1f %% of LDS-active cycles\n"
                        % (100 * sq["SQ_LDS_BANK_CONFLICT"][0] / sq["SQ_LDS_IDX_ACTIVE"][0]))
            st = counters(out, w, "SQSTALL", kern)
            wc = sq.get("SQ_WAVE_CYCLES", (0,))[0]
            if st and wc > 0:
                f.write("SQ stall pass per dispatch (cycle counters as shares of"
                        " SQ_WAVE_CYCLES; instruction counts per wave):\n")
                nw = sq.get("SQ_WAVES", (0,))[0]
                for c in SQ_STALL_COUNTERS:
                    if c not in st:
                        continue
                    if c.startswith("SQ_INSTS_"):
                        f.write("  %-24s %16.0f  %8.0f per wave\n"
                                % (c, st[c][0], st[c][0] / nw if nw else 0))
                    else:
                        f.write("  %-24s %16.0f  %5.1f %%\n" % (c, st[c][0], 100 * st[c][0] / wc))
            if sq.get("SQ_BUSY_CYCLES", (0,))[0] > 0 and "SQ_WAVE_CYCLES" in sq:
                f.write("  mean resident waves per CU: %.1f  (4 x SQ_WAVE_CYCLES / SQ_BUSY_CYCLES"
                        " / %d CUs per shader engine)\n"
                        % (occupancy(sq["SQ_WAVE_CYCLES"][0], sq["SQ_BUSY_CYCLES"][0]),
                           CUS_PER_SE))
            if sq.get("SQ_INSTS_VALU", (0,))[0] > 0 and sq.get("SQ_WAVES", (0,))[0] > 0:
                f.write("  VALU instructions per wave: %.0f; LDS instructions per wave: %.0f\n"
                        % (sq["SQ_INSTS_VALU"][0] / sq["SQ_WAVES"][0],
                           sq.get("SQ_INSTS_LDS", (0,))[0] / sq["SQ_WAVES"][0]))
        print(fname, records["%s/%s" % (kern, w)])
    # Records of workloads not summarised in this call stay as they are (each carries its
    # own source hash, so a stale one is ignored by its reader).
    path = os.path.join(dest, "counters.json")
    merged = {}
    if os.path.exists(path):
        with open(path) as f:
            merged = json.load(f)
    merged.update(records)
    with open(path, "w") as f:
        json.dump(merged, f, indent=1)
    return records


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--out", required=True, help="directory for the raw rocprofv3 outputs")
    ap.add_argument("--workloads", nargs="*", default=list(WORKLOADS))
    ap.add_argument("--write", action="store_true", help="write profiles/ from OUT")
    ap.add_argument("--no-run", action="store_true", help="summarise an existing OUT only")
    args = ap.parse_args()
    os.makedirs(args.out, exist_ok=True)
    if not args.no_run:
        run_passes(args.out, args.workloads)
    if args.write:
        write_summaries(args.out, args.workloads)
    return 0


if __name__ == "__main__":
    sys.exit(main())
