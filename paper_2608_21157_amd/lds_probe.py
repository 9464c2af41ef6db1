"""LDS access patterns of the fused star kernel, for the bank-conflict counters.

``python -m paper_2608_21157_amd.lds_probe`` launches ``stencil_probe_lds`` once per
pattern below (names printed in launch order).  Under
``rocprofv3 --pmc SQ_INSTS_LDS SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE SQ_WAVES`` each
launch's counters then describe one pattern; ``--summarize CSV --write FILE`` turns the
counter file into a table of conflict and active cycles per LDS instruction.

The star patterns are the radius-4 fp32 planes of the fused two-step kernel: the u0
plane is a rectangle 20 vectors wide (the 16-vector tile and two halo vectors each side,
320 bytes per row) and the u1 plane 18 vectors wide (288 bytes).  A tile wave covers 4
rows of 16 vectors; the left/right band wave holds 32 rows of one halo vector each side,
its lanes alternating left and right.
"""
from __future__ import annotations

import argparse
import csv
import ctypes
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
PROBE_LIB = os.path.join(HERE, "libstencil_probe.so")
KERNELS = ("stencil_probe_lds_read_kernel", "stencil_probe_lds_write_kernel")
COUNTERS = ("SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT", "SQ_LDS_IDX_ACTIVE", "SQ_WAVES")

R, TXV, TYW, HXV = 4, 16, 32, 1
W0, W1 = TXV + 4 * HXV, TXV + 2 * HXV          # u0 and u1 rectangle widths in vectors


def _u0(r, v):
    return 16 * ((r + 2 * R) * W0 + (v + 2 * HXV))


def _u1(r, v):
    return 16 * ((r + R) * W1 + (v + HXV))


def _band(cell):
    """Lane l of the left/right band wave: row l // 2, left halo vector for even l."""
    return [cell(l // 2, -1 if l % 2 == 0 else TXV) for l in range(64)]


def patterns():
    """(name, write, 64 byte offsets) in launch order."""
    lanes = range(64)
    p = [
        ("contiguous 1 KiB", 0, [16 * l for l in lanes]),
        ("contiguous 1 KiB, +16 B", 0, [16 * l + 16 for l in lanes]),
        ("4 x 256 B, all at 16 B past a 256 B boundary", 0,
         [1024 * (l // 16) + 16 + 16 * (l % 16) for l in lanes]),
        ("4 x 256 B, the first at +16 B, the rest aligned", 0,
         [1024 * (l // 16) + (16 if l < 16 else 0) + 16 * (l % 16) for l in lanes]),
        ("star tile wave, u0 plane (4 rows x 16, pitch 320 B)", 0,
         [_u0(l // 16, l % 16) for l in lanes]),
        ("star tile wave, u0 plane, x - 1", 0, [_u0(l // 16, l % 16 - 1) for l in lanes]),
        ("star tile wave, u1 plane (4 rows x 16, pitch 288 B)", 0,
         [_u1(l // 16, l % 16) for l in lanes]),
        ("4 rows x 16 at pitch 256 B", 0, [256 * (l // 16) + 16 * (l % 16) for l in lanes]),
        ("4 rows x 16 at pitch 512 B", 0, [512 * (l // 16) + 16 * (l % 16) for l in lanes]),
        ("star left/right band wave, u0 plane", 0, _band(_u0)),
        ("star left/right band wave, u1 plane", 0, _band(_u1)),
        ("one lane per row, pitch 320 B", 0, [320 * l for l in lanes]),
        ("one lane per row, pitch 336 B", 0, [336 * l for l in lanes]),
        ("write: contiguous 1 KiB", 1, [16 * l for l in lanes]),
        ("write: star tile wave, u0 plane", 1, [_u0(l // 16, l % 16) for l in lanes]),
        ("write: star left/right band wave, u0 plane", 1, _band(_u0)),
        ("write: star left/right band wave, u1 plane", 1, _band(_u1)),
        ("write: one lane per row, pitch 320 B", 1, [320 * l for l in lanes]),
        ("write: one lane per row, pitch 336 B", 1, [336 * l for l in lanes]),
    ]
    for name, _, offs in p:
        assert len(offs) == 64 and all(0 <= o <= 65520 and o % 16 == 0 for o in offs), name
    return p


def load():
    if not os.path.exists(PROBE_LIB):
        raise ImportError("libstencil_probe.so is not built (%s)" % PROBE_LIB)
    lib = ctypes.CDLL(PROBE_LIB)
    lib.stencil_probe_lds.argtypes = [ctypes.POINTER(ctypes.c_int32), ctypes.c_int32,
                                      ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                      ctypes.c_void_p]
    lib.stencil_probe_lds.restype = ctypes.c_int
    return lib


def run(iters: int = 500, blocks: int = 1024) -> None:
    """Launch every pattern once on cuda:0, one after the other, printing its name."""
    import torch
    lib = load()
    sink = torch.zeros(1, dtype=torch.float32, device="cuda:0")
    stream = torch.cuda.current_stream()
    for name, write, offs in patterns():
        arr = (ctypes.c_int32 * 64)(*offs)
        st = lib.stencil_probe_lds(arr, write, iters, blocks, sink.data_ptr(),
                                   stream.cuda_stream)
        if st != 0:
            raise RuntimeError("stencil_probe_lds failed (%d) on %s" % (st, name))
        stream.synchronize()
        print(name, flush=True)


def summarize(csv_path: str) -> list:
    """Per pattern, in launch order: conflict and active LDS cycles per instruction."""
    per = {}
    with open(csv_path) as f:
        for row in csv.DictReader(f):
            if not any(k in row["Kernel_Name"] for k in KERNELS):
                continue
            per.setdefault(int(row["Dispatch_Id"]), {})[row["Counter_Name"]] = float(
                row["Counter_Value"])
    pats = patterns()
    if len(per) != len(pats):
        raise ValueError("%d probe dispatches in %s, %d patterns" % (len(per), csv_path,
                                                                     len(pats)))
    out = []
    for (name, write, _), (_, c) in zip(pats, sorted(per.items())):
        insts = c["SQ_INSTS_LDS"]
        out.append({"pattern": name, "write": write,
                    "conflict_per_inst": c["SQ_LDS_BANK_CONFLICT"] / insts,
                    "active_per_inst": c["SQ_LDS_IDX_ACTIVE"] / insts,
                    "conflict_share": c["SQ_LDS_BANK_CONFLICT"] / c["SQ_LDS_IDX_ACTIVE"]})
    return out


def render(rows: list, commands: list) -> str:
    lines = ["# LDS access patterns of the fused star kernel (radius 4, fp32): SQ counters",
             "# per pattern, one launch each (1024 workgroups of 4 waves, 4000 accesses",
             "# per wave).  Commands:"]
    lines += ["#   " + c for c in commands]
    lines += ["", "%-56s %10s %10s %8s" % ("pattern", "conflict", "active", "share"),
              "%-56s %10s %10s %8s" % ("", "per inst", "per inst", "")]
    for r in rows:
        lines.append("%-56s %10.3f %10.3f %7.1f%%" % (r["pattern"], r["conflict_per_inst"],
                                                      r["active_per_inst"],
                                                      100 * r["conflict_share"]))
    return "\n".join(lines) + "\n"


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--summarize", metavar="CSV", help="counter CSV of a rocprofv3 run")
    ap.add_argument("--write", metavar="FILE", help="write the summary here")
    ap.add_argument("--command", action="append", default=[],
                    help="command line to record in the summary (repeatable)")
    args = ap.parse_args(argv)
    if args.summarize:
        text = render(summarize(args.summarize), args.command)
        if args.write:
            with open(args.write, "w") as f:
                f.write(text)
        sys.stdout.write(text)
        return 0
    run()
    return 0


if __name__ == "__main__":
    sys.exit(main())
