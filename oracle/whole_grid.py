"""The oracle over a whole full-size grid, evaluated in independent pieces on several host
threads, and compared with a result at every point.

TEST INFRASTRUCTURE ONLY: used by ``tests/`` and by the ``cpu_baseline`` leg of
``bench.py``.  The HIP library never imports it.

The arithmetic is ``oracle.apply`` unchanged.  This module only decides which sub-grid
each call sees, so that every kept point is computed from exactly the operands it has in
the whole-grid run:

* a batch of volumes splits into its volumes (volume b uses weight set b mod channels and
  its own slice of the coefficient field);
* one volume splits into slabs along its slowest axis (z in 3D, y in 2D).  A slab that
  keeps planes [z0, z1) is evaluated on [z0 - H, z1 + H) with H = radius * steps, the
  reach of ``steps`` iterations:
    - ZERO boundary: the halo is clipped at the grid's faces, where the sub-grid's own
      zero padding is the grid's; at a cut face the sub-grid's padding is wrong, but
      its effect travels at most radius planes per step and never reaches [z0, z1);
    - PERIODIC boundary: the halo planes are taken with wrapped indices, so the sub-grid
      holds the periodic extension; the sub-grid's own wrap along the slab axis only
      touches planes within H of its ends, which are dropped.  x and y keep their
      periodic wrap.  When a slab plus its halo would span the whole axis, the whole
      grid is evaluated as one piece.
Every kept value is therefore bit-identical to the whole-grid oracle's (the same operands
summed in the same order); ``tests/test_whole_grid.py`` checks that on small grids.

``ctypes`` releases the interpreter lock during the oracle's C call, so pieces run in
parallel on a thread pool (no process is forked from a program that may have initialised
the GPU).
"""
from __future__ import annotations

import os
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from . import apply as _oracle_apply

ZERO, PERIODIC = 0, 1


def default_threads() -> int:
    """Host threads for the pieces: the CPUs this process may run on, at most 16."""
    try:
        n = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _split(x: np.ndarray, ndim: int):
    """(batch, dims) of an array shaped (*dims), (batch, *dims) or (N, C, *dims)."""
    if x.ndim == ndim:
        return 1, tuple(x.shape)
    if x.ndim == ndim + 1:
        return x.shape[0], tuple(x.shape[1:])
    if x.ndim == ndim + 2:
        return x.shape[0] * x.shape[1], tuple(x.shape[2:])
    raise ValueError("input rank does not match ndim")


def pieces(x, *, radius: int, boundary: int, steps: int, ndim: int, field=None,
           count: int | None = None):
    """The pieces of a whole-grid evaluation, as dicts with
    ``b`` (volume), ``src`` (plane indices of the sub-grid along the slowest axis, or
    None for the whole volume), ``keep`` (slice of the sub-grid's planes kept) and
    ``dst`` (slice of the volume's planes they fill).  ``count`` is the number of slabs a
    single volume is cut into (default: about two per thread)."""
    batch, dims = _split(x, ndim)
    n0 = dims[0]
    out = []
    if batch > 1:
        for b in range(batch):
            out.append({"b": b, "src": None, "keep": slice(0, n0), "dst": slice(0, n0)})
        return out
    halo = radius * steps
    if count is None:
        count = 2 * default_threads()
        if halo > 0:  # keep a slab at least twice its halo, so at most half is redundant
            count = min(count, max(1, n0 // (2 * halo)))
    count = max(1, min(count, n0))
    length = -(-n0 // count)
    starts = list(range(0, n0, length))
    if boundary == PERIODIC and any(min(z + length, n0) - z + 2 * halo >= n0 for z in starts):
        starts, length = [0], n0
    for z0 in starts:
        z1 = min(z0 + length, n0)
        if z0 == 0 and z1 == n0:
            out.append({"b": 0, "src": None, "keep": slice(0, n0), "dst": slice(0, n0)})
        elif boundary == PERIODIC:
            src = np.arange(z0 - halo, z1 + halo) % n0
            out.append({"b": 0, "src": src, "keep": slice(halo, halo + z1 - z0),
                        "dst": slice(z0, z1)})
        else:
            lo, hi = max(0, z0 - halo), min(n0, z1 + halo)
            out.append({"b": 0, "src": np.arange(lo, hi), "keep": slice(z0 - lo, z1 - lo),
                        "dst": slice(z0, z1)})
    return out


def _volume(a, b: int, batch: int, dims):
    return a.reshape((batch,) + tuple(dims))[b]


def _evaluate_piece(pc, x, w, field, *, shape, radius, boundary, steps, ndim, channels):
    """Oracle values of one piece's kept planes (float64, shape (kept planes, ...))."""
    batch, dims = _split(x, ndim)
    xb = _volume(x, pc["b"], batch, dims)
    kb = None if field is None else _volume(field, pc["b"], batch, dims)
    if pc["src"] is not None:
        xb = xb[pc["src"]]
        kb = None if kb is None else kb[pc["src"]]
    wb = np.asarray(w).reshape(channels, -1)[pc["b"] % channels]
    ref = _oracle_apply(xb, wb, shape=shape, radius=radius, boundary=boundary, steps=steps,
                        field=kb, ndim=ndim, channels=1)
    return ref[pc["keep"]]


def evaluate(x, w, *, shape: int, radius: int, boundary: int = ZERO, steps: int = 1,
             ndim: int, channels: int = 1, field=None, threads: int | None = None,
             count: int | None = None) -> np.ndarray:
    """The whole-grid oracle result assembled from its pieces (float64, ``x``'s shape).
    For grids small enough to hold twice in memory; ``compare`` never assembles."""
    batch, dims = _split(x, ndim)
    out = np.empty((batch,) + tuple(dims), dtype=np.float64)
    kw = dict(shape=shape, radius=radius, boundary=boundary, steps=steps, ndim=ndim,
              channels=channels)
    pcs = pieces(x, radius=radius, boundary=boundary, steps=steps, ndim=ndim, field=field,
                 count=count)

    def work(pc):
        out[pc["b"]][pc["dst"]] = _evaluate_piece(pc, x, w, field, **kw)

    with ThreadPoolExecutor(threads or default_threads()) as ex:
        list(ex.map(work, pcs))
    return out.reshape(x.shape)


def compare(got, x, w, *, shape: int, radius: int, boundary: int = ZERO, steps: int = 1,
            ndim: int, channels: int = 1, field=None, threads: int | None = None,
            count: int | None = None) -> dict:
    """Compare ``got`` (a result shaped like ``x``) with the oracle at every point.

    Returns ``points`` (compared), ``nonfinite`` (values of ``got`` that are NaN or
    infinite), ``max_abs_err``, ``worst`` (flat index into ``x`` of the largest
    error), ``seconds`` (wall time of the evaluation), ``threads`` and ``pieces``."""
    batch, dims = _split(x, ndim)
    g = np.asarray(got).reshape((batch,) + tuple(dims))
    kw = dict(shape=shape, radius=radius, boundary=boundary, steps=steps, ndim=ndim,
              channels=channels)
    pcs = pieces(x, radius=radius, boundary=boundary, steps=steps, ndim=ndim, field=field,
                 count=count)
    plane = int(np.prod(dims[1:])) if len(dims) > 1 else 1
    vol = int(np.prod(dims))

    def work(pc):
        ref = _evaluate_piece(pc, x, w, field, **kw)
        gp = g[pc["b"]][pc["dst"]]
        bad = int(np.count_nonzero(~np.isfinite(gp)))
        err = np.abs(gp.astype(np.float64) - ref)
        if bad:
            err[~np.isfinite(err)] = np.inf
        i = int(np.argmax(err)) if err.size else 0
        worst = float(err.flat[i]) if err.size else 0.0
        flat = pc["b"] * vol + pc["dst"].start * plane + i
        return int(gp.size), bad, worst, flat

    nthreads = threads or default_threads()
    t0 = time.perf_counter()
    with ThreadPoolExecutor(nthreads) as ex:
        res = list(ex.map(work, pcs))
    dt = time.perf_counter() - t0
    worst = max(res, key=lambda r: r[2]) if res else (0, 0, 0.0, 0)
    return {"points": sum(r[0] for r in res), "nonfinite": sum(r[1] for r in res),
            "max_abs_err": worst[2], "worst": worst[3], "seconds": round(dt, 3),
            "threads": nthreads, "pieces": len(pcs)}
