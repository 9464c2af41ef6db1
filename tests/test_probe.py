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
