"""Build the HIP library ``libstencil.so`` for gfx950 with hipcc.

Every HIP/C++ source under ``csrc/`` is compiled to an object in ``_build/`` (in parallel)
and linked into ``libstencil.so`` next to this file; ``csrc/fastcall.c`` becomes the
binding's CPython extension, linked against it.  ``build()`` always recompiles.  A kernel
that uses scratch memory fails the build.
"""
from __future__ import annotations

import concurrent.futures
import os
import re
import shutil
import subprocess
import sys
import sysconfig

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libstencil.so")
PROBE_LIB = os.path.join(HERE, "libstencil_probe.so")
# the CPython extension Plan.run calls stencil_apply through (argument marshalling only)
FASTCALL = os.path.join(HERE, "_fastcall" + (sysconfig.get_config_var("EXT_SUFFIX") or ".so"))
ARCH = "gfx950"

SOURCES = ["abi.cpp", "kernel_generic.hip", "kernel_stream.hip", "kernel_box.hip", "kernel_star.hip",
           "kernel_star_tb.hip", "kernel_star_tbs.hip", "kernel_box2.hip", "kernel_check.hip",
           "noalloc.hip"]

# Packed FP32 instructions are kept out of every kernel (-packed-fp32-ops).
FLAGS = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wextra", "-Wno-unused-parameter",
         "--offload-arch=" + ARCH, "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-ffp-contract=fast", "-I", INCLUDE, "-I", CSRC]


def hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP library cannot be built")


def scratch_kernels(remarks: str) -> list:
    """Kernels that the compiler's resource-usage remarks report with scratch memory
    (private arrays or spills moved out of registers)."""
    out, name = [], None
    for line in remarks.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and int(m.group(1)) > 0:
            out.append((name, int(m.group(1))))
    return out


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    remarks = ["-Rpass-analysis=kernel-resource-usage"] if src.endswith(".hip") else []
    cmd = [hipcc()] + lang + FLAGS + remarks + ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, " ".join(cmd), r.stderr))
    # Every kernel here keeps its queues and accumulators in registers; a kernel that the
    # compiler moved to scratch memory runs an order of magnitude slower, so it is a
    # build error rather than a silent slowdown.
    bad = scratch_kernels(r.stderr)
    if bad:
        raise RuntimeError("%s: kernels using scratch memory: %s" % (
            src, ", ".join("%s (%d B/lane)" % b for b in bad)))
    return obj


PROBE_SOURCES = ["probe_copy.hip", "probe_lds.hip"]


def _link(objs, lib):
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (" ".join(cmd), r.stderr))
    os.replace(tmp, lib)


def build_fastcall() -> str:
    """Compile the CPython extension (gcc) against the built libstencil.so beside it."""
    tmp = FASTCALL + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-D__HIP_PLATFORM_AMD__", "-I", sysconfig.get_paths()["include"], "-I", INCLUDE,
           "-I", "/opt/rocm/include", os.path.join(CSRC, "fastcall.c"), "-L", HERE,
           "-lstencil", "-Wl,-rpath,$ORIGIN", "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("gcc failed for fastcall.c:\n%s\n%s" % (" ".join(cmd), r.stderr))
    os.replace(tmp, FASTCALL)
    return FASTCALL


def build(verbose: bool = False) -> str:
    """Compile and link libstencil.so, the copy probe libstencil_probe.so and the
    binding's CPython extension."""
    os.makedirs(BUILD, exist_ok=True)
    srcs = SOURCES + PROBE_SOURCES
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    _link(objs[: len(SOURCES)], LIB)
    _link(objs[len(SOURCES):], PROBE_LIB)
    build_fastcall()
    if verbose:
        print("built", LIB, PROBE_LIB, "and", FASTCALL)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
