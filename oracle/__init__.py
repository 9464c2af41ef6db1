"""Python access to the fp64 CPU oracle of the stencil operator (``oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py``.  The HIP library and its binding never import it.

Operator (HIERA, experimental setup, paragraph "Case-study protocol"): a zero-padded
cross-correlation with padding R and stride 1, iterated, in FP64; generalised to star and
box offset sets in 2D and 3D, zero or periodic boundaries, an output-indexed coefficient
field and batched volumes with per-channel weights.  ``oracle.c`` states the definition
and the weight order; this module only marshals numpy arrays (promoted to float64) into it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

STAR, BOX = 0, 1
ZERO, PERIODIC = 0, 1

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def compile_source(src: str, dst: str) -> str:
    """gcc -O2 without fast-math or contraction, so the documented sum order is kept."""
    tmp = dst + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", "-std=c11", "-O2", "-fno-fast-math", "-ffp-contract=off",
                           "-fPIC", "-shared", "-Wall", "-Wextra", "-o", tmp, src])
    os.replace(tmp, dst)
    return dst


def build(force: bool = False) -> str:
    """Compile ``oracle.c`` into ``liboracle.so`` (always when ``force``)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        compile_source(_SRC, _LIB)
    return _LIB


def bind(path: str):
    """Load an oracle shared library and declare its entry points."""
    lib = ctypes.CDLL(path)
    i64p = ctypes.POINTER(ctypes.c_int64)
    dp = ctypes.POINTER(ctypes.c_double)
    lib.oracle_num_points.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int]
    lib.oracle_num_points.restype = ctypes.c_int
    lib.oracle_offsets.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                   ctypes.POINTER(ctypes.c_int32)]
    lib.oracle_offsets.restype = ctypes.c_int
    lib.oracle_apply.argtypes = [dp, dp, ctypes.c_int, i64p, ctypes.c_int64, ctypes.c_int,
                                 ctypes.c_int, ctypes.c_int, ctypes.c_int, dp, dp,
                                 ctypes.c_int]
    lib.oracle_apply.restype = ctypes.c_int
    lib.oracle_apply_points.argtypes = [dp, ctypes.c_int, i64p, ctypes.c_int64, ctypes.c_int,
                                        ctypes.c_int, ctypes.c_int, ctypes.c_int, dp, dp,
                                        ctypes.c_int, ctypes.c_int64, i64p, dp]
    lib.oracle_apply_points.restype = ctypes.c_int
    return lib


def _load(lib=None):
    global _lib
    if lib is not None:
        return lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = bind(_LIB)
    return _lib


def num_points(shape: int, ndim: int, radius: int, lib=None) -> int:
    return _load(lib).oracle_num_points(shape, ndim, radius)


def offsets(shape: int, ndim: int, radius: int, lib=None) -> np.ndarray:
    """Offsets (oz, oy, ox) in weight order, shape (npts, 3); oz = 0 in 2D."""
    n = num_points(shape, ndim, radius, lib)
    if n < 0:
        raise ValueError("bad stencil description")
    off = np.zeros((n, 3), dtype=np.int32)
    rc = _load(lib).oracle_offsets(shape, ndim, radius,
                                off.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)))
    if rc != 0:
        raise ValueError("oracle_offsets failed")
    return off


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _dp(a):
    return None if a is None else a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _grid_dims(x: np.ndarray, ndim: int, batch: int):
    """Split an array of shape (batch?, *dims) into (batch, dims)."""
    if x.ndim == ndim:
        return 1, tuple(x.shape)
    if x.ndim == ndim + 1:
        return x.shape[0], tuple(x.shape[1:])
    if x.ndim == ndim + 2:  # (N, C, *dims) conv layout
        return x.shape[0] * x.shape[1], tuple(x.shape[2:])
    raise ValueError("input rank does not match ndim")


def apply(x, w, *, shape: int, radius: int, boundary: int = ZERO, steps: int = 1,
          field=None, ndim: int | None = None, channels: int = 1,
          lib=None) -> np.ndarray:
    """Run the full oracle.  ``x``: (*dims), (batch, *dims) or (N, C, *dims).
    ``w``: (channels, npts) or (npts,).  Returns float64 of ``x``'s shape."""
    x = _f64(x)
    if ndim is None:
        ndim = 3 if x.ndim >= 3 else 2
    batch, dims = _grid_dims(x, ndim, 1)
    w = _f64(w).reshape(channels, -1)
    npts = num_points(shape, ndim, radius, lib)
    if w.shape[1] != npts:
        raise ValueError("expected %d weights per channel, got %d" % (npts, w.shape[1]))
    k = None if field is None else _f64(field)
    if k is not None and k.size != x.size:
        raise ValueError("field must have the input's size")
    out = np.empty_like(x)
    d = (ctypes.c_int64 * 3)(*dims, *([0] * (3 - len(dims))))
    rc = _load(lib).oracle_apply(_dp(x), _dp(out), ndim, d, batch, channels, shape, radius,
                              boundary, _dp(w), _dp(k), steps)
    if rc != 0:
        raise ValueError("oracle_apply rejected its arguments")
    return out


def apply_points(x, w, pts, *, shape: int, radius: int, boundary: int = ZERO, steps: int = 1,
                 field=None, ndim: int | None = None, channels: int = 1,
                 lib=None) -> np.ndarray:
    """Oracle value of ``steps`` steps at selected points.  ``pts``: (n, 4) rows of
    (b, z, y, x), z = 0 in 2D.  Returns float64 of shape (n,)."""
    x = _f64(x)
    if ndim is None:
        ndim = 3 if x.ndim >= 3 else 2
    batch, dims = _grid_dims(x, ndim, 1)
    w = _f64(w).reshape(channels, -1)
    k = None if field is None else _f64(field)
    pts = np.ascontiguousarray(pts, dtype=np.int64).reshape(-1, 4)
    vals = np.empty(pts.shape[0], dtype=np.float64)
    d = (ctypes.c_int64 * 3)(*dims, *([0] * (3 - len(dims))))
    rc = _load(lib).oracle_apply_points(_dp(x), ndim, d, batch, channels, shape, radius, boundary,
                                     _dp(w), _dp(k), steps, pts.shape[0],
                                     pts.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                     _dp(vals))
    if rc != 0:
        raise ValueError("oracle_apply_points rejected its arguments")
    return vals
