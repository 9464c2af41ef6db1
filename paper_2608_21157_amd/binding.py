"""ctypes binding of ``libstencil.so`` (the C ABI declared in ``include/stencil.h``).

Argument marshalling only: every step of the operator runs in the library's HIP kernels.
The functions keep the C names (``stencil_plan``, ``stencil_apply``, ``stencil_destroy``,
...) and raise ``StencilError`` on a non-OK status.  ``Plan`` and ``apply`` are thin
conveniences over them for torch tensors (torch supplies device memory and streams);
``Plan.run`` calls ``stencil_apply`` through the small CPython extension ``_fastcall``
(built from ``csrc/fastcall.c`` against the same library), which converts ten integers
per call where ctypes would convert ten objects.

The library must have been built (``python -m paper_2608_21157_amd.build``); there is no
fallback: loading fails loudly when it is missing.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libstencil.so")

# enums of stencil.h
OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_MISMATCH, ERR_ALIAS, ERR_NO_MEMORY, ERR_HIP = range(7)
F32, F64 = 0, 1
STAR, BOX = 0, 1
ZERO, PERIODIC = 0, 1
VARIANT_AUTO, VARIANT_GENERIC, VARIANT_STREAM = 0, 1, 2
VARIANT_NAMES = {VARIANT_GENERIC: "generic", VARIANT_STREAM: "stream"}

EXPORTED = ("stencil_plan", "stencil_apply", "stencil_destroy", "stencil_plan_query",
            "stencil_num_points", "stencil_status_str", "stencil_last_error", "stencil_tune",
            "stencil_apply_noalloc")
NOALLOC_WEIGHT_BYTES = 64 * 1024       # STENCIL_NOALLOC_WEIGHT_BYTES
NOALLOC_GRID_BYTES = 64 * 1024 * 1024  # STENCIL_NOALLOC_GRID_BYTES
TUNE_MAX_CANDIDATES = 20


class StencilDesc(ctypes.Structure):
    _fields_ = [("ndim", ctypes.c_int32), ("dims", ctypes.c_int64 * 3),
                ("batch", ctypes.c_int64), ("channels", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("shape", ctypes.c_int32),
                ("radius", ctypes.c_int32), ("boundary", ctypes.c_int32),
                ("has_coeff_field", ctypes.c_int32), ("variant", ctypes.c_int32),
                ("temporal_depth", ctypes.c_int32), ("tile", ctypes.c_int32),
                ("grid_scale", ctypes.c_int32)]


class StencilPlanInfo(ctypes.Structure):
    _fields_ = [("variant", ctypes.c_int32), ("temporal_depth", ctypes.c_int32),
                ("scratch_bytes", ctypes.c_int64), ("kernel", ctypes.c_char_p),
                ("tile", ctypes.c_int32), ("grid_scale", ctypes.c_int32)]


class StencilTuneEntry(ctypes.Structure):
    _fields_ = [("variant", ctypes.c_int32), ("temporal_depth", ctypes.c_int32),
                ("tile", ctypes.c_int32), ("grid_scale", ctypes.c_int32),
                ("valid", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("max_abs_err", ctypes.c_double), ("ms", ctypes.c_double)]


class StencilTuneReport(ctypes.Structure):
    _fields_ = [("count", ctypes.c_int32), ("chosen", ctypes.c_int32),
                ("tolerance", ctypes.c_double),
                ("entry", StencilTuneEntry * TUNE_MAX_CANDIDATES)]


class StencilError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(detail or "status %d" % status)
        self.status = status


_lib = None
_NO_STREAM = object()   # Plan._sh_obj before the first run: matches no argument, not even None
_fast_apply = None   # _fastcall.apply: stencil_apply with integer arguments, for Plan.run


def load():
    """Load ``libstencil.so`` and declare its signatures (raises if it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("libstencil.so is not built (%s); run "
                          "`python -m paper_2608_21157_amd.build` first" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    vp = ctypes.c_void_p
    lib.stencil_plan.argtypes = [ctypes.POINTER(StencilDesc), ctypes.POINTER(vp)]
    lib.stencil_plan.restype = ctypes.c_int
    lib.stencil_apply.argtypes = [vp, vp, vp, ctypes.POINTER(ctypes.c_int64), vp, vp,
                                  ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, vp]
    lib.stencil_apply.restype = ctypes.c_int
    lib.stencil_apply_noalloc.argtypes = lib.stencil_apply.argtypes
    lib.stencil_apply_noalloc.restype = ctypes.c_int
    lib.stencil_destroy.argtypes = [vp]
    lib.stencil_destroy.restype = ctypes.c_int
    lib.stencil_plan_query.argtypes = [vp, ctypes.POINTER(StencilPlanInfo)]
    lib.stencil_plan_query.restype = ctypes.c_int
    lib.stencil_num_points.argtypes = [ctypes.c_int32] * 3
    lib.stencil_num_points.restype = ctypes.c_int32
    lib.stencil_status_str.argtypes = [ctypes.c_int]
    lib.stencil_status_str.restype = ctypes.c_char_p
    lib.stencil_last_error.argtypes = []
    lib.stencil_last_error.restype = ctypes.c_char_p
    lib.stencil_tune.argtypes = [vp, vp, vp, ctypes.POINTER(ctypes.c_int64), vp, vp,
                                 ctypes.c_int32, ctypes.c_double, ctypes.c_int32, vp,
                                 ctypes.POINTER(StencilTuneReport)]
    lib.stencil_tune.restype = ctypes.c_int
    global _fast_apply
    # linked against libstencil.so by name with an $ORIGIN run path: the loader finds the
    # library loaded above (same file), so both share one set of plans and error state
    from . import _fastcall
    _fast_apply = _fastcall.apply
    _lib = lib
    return lib


def _check(status: int) -> None:
    if status != OK:
        raise StencilError(status, load().stencil_last_error().decode())


# ------------------------------------------------------------------ C names, marshalled

def stencil_plan(desc: StencilDesc) -> int:
    h = ctypes.c_void_p()
    _check(load().stencil_plan(ctypes.byref(desc), ctypes.byref(h)))
    return h.value


def stencil_apply(plan: int, inp: int, out: int, dims, coeffs, coeff_field: int | None,
                  radius: int, boundary: int, steps: int, stream: int | None) -> None:
    """``inp``/``out``/``coeff_field``: device addresses; ``coeffs``: a host buffer (numpy
    array or ctypes pointer) of the plan's dtype; ``stream``: a hipStream_t handle."""
    d = dims if isinstance(dims, ctypes.Array) else _dims3(dims)
    cp = coeffs.ctypes.data if hasattr(coeffs, "ctypes") else coeffs
    _check(load().stencil_apply(plan, inp, out, d, cp, coeff_field, radius, boundary, steps,
                                stream))


def stencil_apply_noalloc(plan: int, inp: int, out: int, dims, coeffs,
                          coeff_field: int | None, radius: int, boundary: int, steps: int,
                          stream: int | None) -> None:
    """``stencil_apply`` through the library's static scratch (no device allocation);
    arguments as ``stencil_apply``."""
    d = dims if isinstance(dims, ctypes.Array) else _dims3(dims)
    cp = coeffs.ctypes.data if hasattr(coeffs, "ctypes") else coeffs
    _check(load().stencil_apply_noalloc(plan, inp, out, d, cp, coeff_field, radius, boundary,
                                        steps, stream))


def _dims3(dims) -> ctypes.Array:
    return (ctypes.c_int64 * 3)(*(list(dims) + [0] * (3 - len(dims))))


def stencil_tune(plan: int, inp: int, out: int, dims, coeffs, coeff_field: int | None,
                 steps: int, tolerance: float, reps: int, stream: int | None,
                 report: StencilTuneReport | None = None) -> None:
    """Arguments as ``stencil_apply`` plus the tolerance (< 0: the library's default),
    the timed calls per candidate (0: 5) and an optional report to fill."""
    d = (ctypes.c_int64 * 3)(*(list(dims) + [0] * (3 - len(dims))))
    cp = coeffs.ctypes.data if hasattr(coeffs, "ctypes") else coeffs
    rp = ctypes.byref(report) if report is not None else None
    _check(load().stencil_tune(plan, inp, out, d, cp, coeff_field, steps, float(tolerance),
                               reps, stream, rp))


def stencil_destroy(plan: int | None) -> None:
    _check(load().stencil_destroy(plan))


def stencil_plan_query(plan: int) -> StencilPlanInfo:
    info = StencilPlanInfo()
    _check(load().stencil_plan_query(plan, ctypes.byref(info)))
    return info


def stencil_num_points(shape: int, ndim: int, radius: int) -> int:
    return load().stencil_num_points(shape, ndim, radius)


def stencil_status_str(status: int) -> str:
    return load().stencil_status_str(status).decode()


def stencil_last_error() -> str:
    return load().stencil_last_error().decode()


# ------------------------------------------------------------------ torch conveniences

def make_desc(ndim, dims, *, batch=1, channels=1, dtype=F32, shape=STAR, radius=1,
              boundary=ZERO, has_coeff_field=False, variant=VARIANT_AUTO,
              temporal_depth=0, tile=0, grid_scale=0) -> StencilDesc:
    d = StencilDesc()
    d.ndim = ndim
    for i, v in enumerate(list(dims)[:3]):
        d.dims[i] = int(v)
    d.batch, d.channels, d.dtype, d.shape = int(batch), int(channels), int(dtype), int(shape)
    d.radius, d.boundary, d.has_coeff_field = int(radius), int(boundary), int(bool(has_coeff_field))
    d.variant, d.temporal_depth = int(variant), int(temporal_depth)
    d.tile, d.grid_scale = int(tile), int(grid_scale)
    return d


class Plan:
    """Owns a ``stencil_plan_t``; ``run`` calls ``stencil_apply`` on torch tensors.

    ``run`` validates its tensors and weight array once per new object: the dtype is the
    plan's, the element count is batch * volume, tensors are contiguous CUDA tensors on
    one device, and the weights are a C-contiguous numpy array of channels * npoints
    values of the plan's dtype.  A failed check raises ``ValueError`` before the library
    is called.  The objects last validated are held until another one is passed (or the
    plan is closed), so an unchanged object is not checked again; resizing a validated
    tensor in place between calls is not detected.  Weight values changed in place are
    still seen: the library compares the weights' bytes on every call.  A Plan is used
    from one thread at a time (its cached arguments and the plan's buffers are shared
    state); separate Plans may run on separate threads and streams."""

    def __init__(self, desc: StencilDesc):
        self.desc = desc
        self.handle = stencil_plan(desc)
        self.dims = tuple(desc.dims[i] for i in range(desc.ndim))
        self._dims_c = _dims3(self.dims)  # built once: run() is on the latency path
        self._dims_addr = ctypes.addressof(self._dims_c)
        self._numel = int(desc.batch)
        for d in self.dims:
            self._numel *= int(d)
        self._ncoeffs = int(desc.channels) * stencil_num_points(desc.shape, desc.ndim,
                                                                desc.radius)
        self._stream = None               # last stream run on (close() waits for it)
        self._seen = (None, None, None, None)   # x, y, field, coeffs last validated
        self._sh_obj = _NO_STREAM         # stream argument whose handle is in _sh
        self._sh = 0                      # that stream's handle (0: the null stream)
        self._fast = _fast_apply
        self._pc = 0                      # address of the weights last validated
        self._radius = int(desc.radius)
        self._boundary = int(desc.boundary)

    def info(self) -> StencilPlanInfo:
        return stencil_plan_query(self.handle)

    def _validate(self, x, y, coeffs, field) -> None:
        import numpy as np
        import torch
        want = torch.float32 if self.desc.dtype == F32 else torch.float64
        named = [("x", x), ("y", y)] + ([("field", field)] if field is not None else [])
        for name, t in named:
            if not isinstance(t, torch.Tensor):
                raise ValueError("%s must be a torch tensor" % name)
            if t.dtype != want:
                raise ValueError("%s has dtype %s, the plan computes in %s" % (name, t.dtype,
                                                                              want))
            if t.numel() != self._numel:
                raise ValueError("%s has %d elements, the plan needs batch * volume = %d"
                                 % (name, t.numel(), self._numel))
            if not t.is_contiguous():
                raise ValueError("%s must be contiguous" % name)
        if (field is not None) != bool(self.desc.has_coeff_field):
            raise ValueError("the plan needs a coefficient field" if self.desc.has_coeff_field
                             else "the plan has no coefficient field")
        npdt = np.float32 if self.desc.dtype == F32 else np.float64
        if not isinstance(coeffs, np.ndarray):
            raise ValueError("coeffs must be a numpy array on the host")
        if coeffs.dtype != npdt:
            raise ValueError("coeffs has dtype %s, the plan computes in %s" % (
                coeffs.dtype, np.dtype(npdt)))
        if coeffs.size != self._ncoeffs:
            raise ValueError("coeffs has %d values, the plan needs channels * npoints = %d"
                             % (coeffs.size, self._ncoeffs))
        if not coeffs.flags.c_contiguous:
            raise ValueError("coeffs must be C-contiguous")
        devs = {t.device for _, t in named}
        if any(d.type != "cuda" for d in devs) or len(devs) != 1:
            raise ValueError("x, y (and field) must be CUDA tensors on one device")
        self._seen = (x, y, field, coeffs)
        self._pc = coeffs.ctypes.data

    def run(self, x, y, coeffs, *, steps: int, field=None, stream=None) -> None:
        seen = self._seen
        if x is not seen[0] or y is not seen[1] or field is not seen[2] or coeffs is not seen[3]:
            self._validate(x, y, coeffs, field)
        if stream is not self._sh_obj:
            if stream is None:
                import torch
                stream = torch.cuda.current_stream()
            self._sh = (stream.cuda_stream if hasattr(stream, "cuda_stream") else stream) or 0
            self._sh_obj = stream
        self._stream = stream
        st = self._fast(self.handle or 0, x.data_ptr(), y.data_ptr(), self._dims_addr,
                        self._pc, 0 if field is None else field.data_ptr(), self._radius,
                        self._boundary, steps, self._sh)
        if st:
            _check(st)

    def tune(self, x, y, coeffs, *, steps: int, field=None, tolerance: float = -1.0,
             reps: int = 0, stream=None) -> dict:
        """``stencil_tune`` on torch tensors: fixes the fastest candidate that passes the
        validity gate in this plan and leaves its result in ``y``.  Returns the report as
        a dict: ``tolerance``, ``chosen`` (index) and ``candidates`` (list of dicts)."""
        import torch
        self._validate(x, y, coeffs, field)
        if stream is None:
            stream = torch.cuda.current_stream()
        sh = stream.cuda_stream if hasattr(stream, "cuda_stream") else stream
        self._stream = stream
        rep = StencilTuneReport()
        stencil_tune(self.handle, x.data_ptr(), y.data_ptr(), self.dims, coeffs,
                     None if field is None else field.data_ptr(), steps, tolerance, reps, sh,
                     rep)
        cands = [{"variant": VARIANT_NAMES.get(e.variant, str(e.variant)),
                  "temporal_depth": e.temporal_depth, "tile": e.tile,
                  "grid_scale": e.grid_scale, "valid": bool(e.valid),
                  "max_abs_err": e.max_abs_err, "ms": e.ms}
                 for e in rep.entry[: rep.count]]
        return {"tolerance": rep.tolerance, "chosen": rep.chosen, "candidates": cands}

    def close(self) -> None:
        """Wait for the last stream this plan ran on, then free the plan."""
        self._seen = (None, None, None, None)
        self._sh_obj = _NO_STREAM
        if self.handle:
            if self._stream is not None and hasattr(self._stream, "synchronize"):
                self._stream.synchronize()
            stencil_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def apply(x, y, coeffs, *, shape: int, radius: int, boundary: int = ZERO, steps: int = 1,
          field=None, ndim: int | None = None, channels: int = 1, variant: int = VARIANT_AUTO,
          temporal_depth: int = 0, stream=None) -> None:
    """One-shot: plan, apply and destroy.  ``x``, ``y`` (and ``field``): contiguous CUDA
    tensors of shape (*dims), (batch, *dims) or (N, C, *dims), float32 or float64;
    ``coeffs``: host numpy array (channels, npoints) of the same dtype."""
    import numpy as np
    import torch
    if not (x.is_cuda and y.is_cuda and x.is_contiguous() and y.is_contiguous()):
        raise ValueError("x and y must be contiguous device tensors")
    if x.dtype != y.dtype or x.shape != y.shape:
        raise ValueError("x and y must have the same dtype and shape")
    if field is not None and (not field.is_cuda or not field.is_contiguous()
                              or field.dtype != x.dtype or field.shape != x.shape):
        raise ValueError("field must be a contiguous device tensor shaped like x")
    dt = {torch.float32: F32, torch.float64: F64}.get(x.dtype)
    if dt is None:
        raise ValueError("float32 or float64 tensors only")
    if ndim is None:
        ndim = 3 if x.dim() >= 3 else 2
    lead = x.shape[: x.dim() - ndim]
    batch = int(np.prod(lead)) if len(lead) else 1
    c = np.ascontiguousarray(coeffs, dtype=np.float32 if dt == F32 else np.float64)
    desc = make_desc(ndim, x.shape[x.dim() - ndim:], batch=batch, channels=channels, dtype=dt,
                     shape=shape, radius=radius, boundary=boundary,
                     has_coeff_field=field is not None, variant=variant,
                     temporal_depth=temporal_depth)
    p = Plan(desc)
    try:
        p.run(x, y, c, steps=steps, field=field, stream=stream)
    finally:
        p.close()
