"""The C ABI from plain C: ``tests/c_consumer.c`` includes ``include/stencil.h`` as a C99
translation unit (gcc, not hipcc), links ``libstencil.so`` and runs host-side checks of
every entry point (see the C file).  This shows the boundary carries no C++ or torch type
and that its symbols resolve for a C caller."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIBDIR = os.path.join(ROOT, "paper_2608_21157_amd")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc is not available")
def test_c_consumer(tmp_path):
    if not os.path.exists(os.path.join(LIBDIR, "libstencil.so")):
        pytest.fail("libstencil.so is not built")
    exe = str(tmp_path / "c_consumer")
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
           os.path.join(ROOT, "tests", "c_consumer.c"), "-L", LIBDIR, "-lstencil",
           "-Wl,-rpath," + LIBDIR, "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout
