"""The HBM copy probe (``libstencil_probe.so``): argument checks on the CPU, exact copies of
ragged sizes on the GPU.  The probe is measurement infrastructure (the copy ceiling and the
calibration of hardware byte counters); it has no part in the stencil path."""
import ctypes
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PROBE = os.path.join(ROOT, "paper_2608_21157_amd", "libstencil_probe.so")
A, B_ = 0x7F0000000000, 0x7F0100000000  # aligned placeholders, never dereferenced


def probe():
    if not os.path.exists(PROBE):
        pytest.fail("%s is not built (python -m paper_2608_21157_amd.build)" % PROBE)
    lib = ctypes.CDLL(PROBE)
    lib.stencil_probe_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                       ctypes.c_void_p]
    lib.stencil_probe_copy.restype = ctypes.c_int
    lib.stencil_probe_triad.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_int64, ctypes.c_void_p]
    lib.stencil_probe_triad.restype = ctypes.c_int
    return lib


def test_probe_rejects_invalid_arguments_before_any_hip_call():
    lib = probe()
    assert lib.stencil_probe_copy(None, B_, 64, None) == 1
    assert lib.stencil_probe_copy(A, None, 64, None) == 1
    assert lib.stencil_probe_copy(A, B_, -16, None) == 1
    assert lib.stencil_probe_copy(A, B_, 24, None) == 1          # not a multiple of 16
    assert lib.stencil_probe_copy(A + 8, B_, 64, None) == 1      # misaligned source
    assert lib.stencil_probe_copy(A, B_ + 4, 64, None) == 1      # misaligned destination
    assert lib.stencil_probe_copy(A, B_, 0, None) == 0           # nothing to do, no launch


def test_triad_rejects_invalid_arguments_before_any_hip_call():
    lib = probe()
    C = 0x7F0200000000
    assert lib.stencil_probe_triad(None, B_, C, 64, None) == 1
    assert lib.stencil_probe_triad(A, None, C, 64, None) == 1
    assert lib.stencil_probe_triad(A, B_, None, 64, None) == 1
    assert lib.stencil_probe_triad(A, B_, C, -16, None) == 1
    assert lib.stencil_probe_triad(A, B_, C, 40, None) == 1       # not a multiple of 16
    assert lib.stencil_probe_triad(A + 4, B_, C, 64, None) == 1   # misaligned input
    assert lib.stencil_probe_triad(A, B_, C + 8, 64, None) == 1   # misaligned output
    assert lib.stencil_probe_triad(A, B_, C, 0, None) == 0        # nothing to do, no launch


@pytest.mark.gpu
@pytest.mark.parametrize("nbytes", [16, 4096, 4096 + 16, 3 * 4096 + 48, 1 << 20,
                                    (1 << 24) + 4080])
def test_probe_copies_exactly(nbytes):
    import torch
    lib = probe()
    src = torch.randint(0, 256, (nbytes + 64,), dtype=torch.uint8, device="cuda:0")
    dst = torch.zeros(nbytes + 64, dtype=torch.uint8, device="cuda:0")
    stream = torch.cuda.current_stream()
    assert lib.stencil_probe_copy(src.data_ptr(), dst.data_ptr(), nbytes,
                                  stream.cuda_stream) == 0
    stream.synchronize()
    assert torch.equal(dst[:nbytes], src[:nbytes])
    assert int(dst[nbytes:].abs().sum()) == 0   # nothing written past the end


@pytest.mark.gpu
@pytest.mark.parametrize("nbytes", [16, 4096 + 16, (1 << 22) + 48])
def test_triad_multiplies_exactly(nbytes):
    import torch
    lib = probe()
    n = nbytes // 4
    a = torch.rand(n + 16, device="cuda:0")
    b = torch.rand(n + 16, device="cuda:0")
    dst = torch.zeros(n + 16, device="cuda:0")
    stream = torch.cuda.current_stream()
    assert lib.stencil_probe_triad(a.data_ptr(), b.data_ptr(), dst.data_ptr(), nbytes,
                                   stream.cuda_stream) == 0
    stream.synchronize()
    assert torch.equal(dst[:n], a[:n] * b[:n])    # one fp32 product, correctly rounded
    assert int((dst[n:] != 0).sum()) == 0         # nothing written past the end


# ------------------------------------------------------------------ the LDS pattern probe

def test_lds_probe_rejects_invalid_arguments_before_any_hip_call():
    from paper_2608_21157_amd import lds_probe
    lib = lds_probe.load()
    ok = (ctypes.c_int32 * 64)(*[16 * i for i in range(64)])
    sink = A
    assert lib.stencil_probe_lds(None, 0, 1, 1, sink, None) == 1
    assert lib.stencil_probe_lds(ok, 2, 1, 1, sink, None) == 1
    assert lib.stencil_probe_lds(ok, 0, 0, 1, sink, None) == 1
    assert lib.stencil_probe_lds(ok, 0, 1, 0, sink, None) == 1
    assert lib.stencil_probe_lds(ok, 0, (1 << 20) + 1, 1, sink, None) == 1
    assert lib.stencil_probe_lds(ok, 0, 1, 1, None, None) == 1
    for bad in (-16, 8, 65536):
        arr = (ctypes.c_int32 * 64)(*[16 * i for i in range(64)])
        arr[17] = bad
        assert lib.stencil_probe_lds(arr, 1, 1, 1, sink, None) == 1


def test_lds_probe_patterns_are_the_kernel_layout():
    """The star patterns follow the fused kernel's u0/u1 rectangles at radius 4, fp32:
    rows of 20 and 18 vectors, origins 8 rows / 2 vectors and 4 rows / 1 vector out."""
    from paper_2608_21157_amd import lds_probe as L
    pats = {name: (w, offs) for name, w, offs in L.patterns()}
    assert len(pats) == len(L.patterns())                      # names are unique
    _, tile = pats["star tile wave, u0 plane (4 rows x 16, pitch 320 B)"]
    assert tile[0] == 16 * (8 * 20 + 2) and tile[16] - tile[0] == 320 and tile[1] - tile[0] == 16
    _, u1 = pats["star tile wave, u1 plane (4 rows x 16, pitch 288 B)"]
    assert u1[0] == 16 * (4 * 18 + 1) and u1[16] - u1[0] == 288
    _, band = pats["star left/right band wave, u0 plane"]
    assert band[0] == 16 * (8 * 20 + 1) and band[1] == 16 * (8 * 20 + 18)
    assert band[2] - band[0] == 320


def test_lds_probe_summary_from_a_counter_file(tmp_path):
    from paper_2608_21157_amd import lds_probe as L
    pats = L.patterns()
    path = tmp_path / "c.csv"
    cols = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]
    with open(path, "w") as f:
        f.write(",".join(cols) + "\n")
        f.write("1,other_kernel,SQ_INSTS_LDS,5\n")
        for i, (_, w, _) in enumerate(pats):
            k = L.KERNELS[w]
            for name, val in (("SQ_INSTS_LDS", 100), ("SQ_LDS_BANK_CONFLICT", 10 * i),
                              ("SQ_LDS_IDX_ACTIVE", 700 + 10 * i), ("SQ_WAVES", 4)):
                f.write("%d,%s,%s,%g\n" % (i + 2, k, name, val))
    rows = L.summarize(str(path))
    assert [r["pattern"] for r in rows] == [p[0] for p in pats]
    assert rows[3]["conflict_per_inst"] == pytest.approx(0.3)
    assert rows[3]["active_per_inst"] == pytest.approx(7.3)
    assert rows[3]["conflict_share"] == pytest.approx(30 / 730)
    assert "pattern" in L.render(rows, ["cmd"])


@pytest.mark.gpu
def test_lds_probe_runs_every_pattern(capsys):
    from paper_2608_21157_amd import lds_probe as L
    L.run(iters=2, blocks=8)
    printed = capsys.readouterr().out.splitlines()
    assert printed == [p[0] for p in L.patterns()]
