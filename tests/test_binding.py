"""Plan.run's argument checks, on the CPU: each wrong tensor or weight array raises
ValueError before the library is called (CPU tensors reach the device check last, so
every other check can be exercised without a GPU)."""
import os

import numpy as np
import pytest
import torch

from paper_2608_21157_amd import binding as B


def plan(field=False, dtype=B.F32, channels=1, batch=1):
    return B.Plan(B.make_desc(3, (4, 5, 8), batch=batch, channels=channels, dtype=dtype,
                              shape=B.BOX, radius=1, has_coeff_field=field))


def good(dtype=torch.float32, batch=1):
    return torch.zeros((batch, 4, 5, 8) if batch > 1 else (4, 5, 8), dtype=dtype)


W27 = np.zeros(27, dtype=np.float32)


def raises(p, msg, *args, **kw):
    with pytest.raises(ValueError, match=msg):
        p.run(*args, steps=1, **kw)


def test_valid_cpu_tensors_stop_at_the_device_check():
    p = plan()
    raises(p, "CUDA tensors", good(), good(), W27)
    p.close()


def test_dtype_count_and_layout_of_the_tensors():
    p = plan()
    raises(p, "dtype torch.float64", good(torch.float64), good(), W27)
    raises(p, "y has dtype", good(), good(torch.float64), W27)
    raises(p, "x has 159 elements", good().flatten()[1:], good(), W27)
    raises(p, "y has 320 elements", good(), torch.zeros(320), W27)
    raises(p, "x must be contiguous", good().transpose(1, 2), good(), W27)
    raises(p, "x must be a torch tensor", good().numpy(), good(), W27)
    p.close()


def test_batch_counts_every_volume():
    p = plan(batch=3, channels=3)
    w = np.zeros((3, 27), dtype=np.float32)
    raises(p, "x has 160 elements, the plan needs batch \\* volume = 480", good(), good(), w)
    raises(p, "CUDA tensors", good(batch=3), good(batch=3), w)
    raises(p, "coeffs has 27 values, the plan needs channels \\* npoints = 81",
           good(batch=3), good(batch=3), W27)
    p.close()


def test_weights_array():
    p = plan()
    raises(p, "coeffs has dtype float64", good(), good(), W27.astype(np.float64))
    raises(p, "coeffs has 26 values", good(), good(), W27[:26])
    raises(p, "C-contiguous", good(), good(), np.zeros(54, dtype=np.float32)[::2])
    raises(p, "numpy array", good(), good(), list(W27))
    p.close()
    p = plan(dtype=B.F64)
    raises(p, "coeffs has dtype float32", good(torch.float64), good(torch.float64), W27)
    p.close()


def test_coefficient_field_presence_and_shape():
    p = plan(field=True)
    raises(p, "needs a coefficient field", good(), good(), W27)
    raises(p, "field has dtype", good(), good(), W27, field=good(torch.float64))
    raises(p, "field has 159 elements", good(), good(), W27, field=good().flatten()[1:])
    raises(p, "CUDA tensors", good(), good(), W27, field=good())
    p.close()
    p = plan()
    raises(p, "has no coefficient field", good(), good(), W27, field=good())
    p.close()


def test_a_failed_check_is_repeated_for_the_same_objects():
    """Nothing is remembered from a failed check: the same objects fail again."""
    p = plan()
    x, y = good(), good()
    for _ in range(2):
        raises(p, "CUDA tensors", x, y, W27)
    p.close()


# ------------------------------------------------------------------ the _fastcall extension

def test_fastcall_shares_the_library_loaded_by_ctypes():
    """The extension resolves libstencil.so to the file ctypes loaded: one copy is mapped,
    so plans made through ctypes are valid handles for it and errors land in one place."""
    B.load()
    from paper_2608_21157_amd import _fastcall
    maps = [ln.split()[-1] for ln in open("/proc/self/maps") if ln.rstrip().endswith(".so")]
    stencil = {m for m in maps if os.path.basename(m) == "libstencil.so"}
    assert stencil == {os.path.realpath(B.LIB_PATH)}
    assert any(os.path.basename(m).startswith("_fastcall.") for m in maps)
    assert _fastcall.apply is B._fast_apply


def test_fastcall_argument_checks():
    from paper_2608_21157_amd import _fastcall
    with pytest.raises(TypeError, match="exactly 10"):
        _fastcall.apply(0, 0, 0)
    with pytest.raises(TypeError):
        _fastcall.apply("plan", 0, 0, 0, 0, 0, 1, 0, 1, 0)
    with pytest.raises(OverflowError):
        _fastcall.apply(0, 0, 0, 0, 0, 0, 1 << 40, 0, 1, 0)
    with pytest.raises(OverflowError):
        _fastcall.apply(0, 0, 0, 0, 0, 0, 1, 0, -(1 << 33), 0)
    with pytest.raises(OverflowError):
        _fastcall.apply(1 << 70, 0, 0, 0, 0, 0, 1, 0, 1, 0)


def test_fastcall_reaches_the_library_checks():
    """Each status of stencil_apply's host checks comes back through the extension as it
    does through ctypes (None and 0 both mean NULL)."""
    import ctypes
    h = B.stencil_plan(B.make_desc(3, (4, 5, 8), shape=B.BOX, radius=1))
    try:
        from paper_2608_21157_amd import _fastcall
        d = (ctypes.c_int64 * 3)(4, 5, 8)
        da = ctypes.addressof(d)
        inp, out = 1 << 20, 1 << 24
        ok = (h, inp, out, da, W27.ctypes.data, None, 1, B.ZERO, 1, None)

        def st(**kw):
            args = list(ok)
            names = ("plan", "inp", "out", "dims", "coeffs", "field", "radius", "boundary",
                     "steps", "stream")
            for k, v in kw.items():
                args[names.index(k)] = v
            return _fastcall.apply(*args)

        assert st(plan=0) == B.ERR_INVALID_ARG
        assert st(plan=None) == B.ERR_INVALID_ARG
        assert st(inp=0) == B.ERR_INVALID_ARG
        assert st(dims=None) == B.ERR_INVALID_ARG
        assert st(steps=-1) == B.ERR_INVALID_ARG
        assert st(radius=2) == B.ERR_MISMATCH
        assert st(boundary=B.PERIODIC) == B.ERR_MISMATCH
        assert st(field=1 << 28) == B.ERR_MISMATCH
        assert st(out=inp) == B.ERR_ALIAS
        if not torch.cuda.is_available():
            assert st() == B.ERR_HIP
            assert "hipGetDevice" in B.stencil_last_error()
    finally:
        B.stencil_destroy(h)


def test_run_resolves_the_stream_argument_on_every_change():
    """Plan.run keeps the last stream's handle; another object, a raw handle or None
    (torch's current stream) is resolved again. The library call is replaced by a recorder
    and the tensors are marked validated, so this runs without a GPU."""
    p = plan()
    x, y = good(), good()
    p._seen = (x, y, None, W27)
    got = []
    p._fast = lambda *a: got.append(a[-1]) or 0

    class S:
        def __init__(self, h):
            self.cuda_stream = h

    s1, s2 = S(111), S(222)
    for stream in (s1, s1, s2, 333, None, s1):
        if stream is None:
            if torch.cuda.is_available():
                continue
            with pytest.raises(Exception):   # no GPU: torch cannot name a current stream
                p.run(x, y, W27, steps=1)
            continue
        p.run(x, y, W27, steps=1, stream=stream)
    assert got == [111, 111, 222, 333, 111]
    p._fast = B._fast_apply
    p._seen = (None, None, None, None)
    p.close()
