"""Seeded synthetic workloads for the stencil operator.

This module generates inputs only: grids, weight vectors and coefficient fields, as numpy
arrays on the host.  It contains none of the operator's arithmetic and imports neither
the HIP binding nor the oracle; the same arrays are handed to both.

Every array comes from ``numpy.random.Generator(PCG64(seed))`` with a fixed draw order
per workload: input first, then weights, then the coefficient field.

Workloads (the paper measures one stencil, a 2D box of radius 3 on a 10240 x 10240 FP64
grid, iterated 10,240 times -- HIERA, experimental setup, "Case-study protocol"; the five
numbered ones below widen that operator to 3D, stars, periodic boundaries, a coefficient
field and batched channels):

  c1  2D 5-point Laplacian, R=1, weights centre -1, neighbours 0.25; 256x256 fp32;
      ZERO boundary; 1 step; input i.i.d. U[-1,1].
  c2  3D 7-point star, R=1, centre 0.4, neighbours 0.1; 256^3 fp32; ZERO; 10 steps;
      input i.i.d. U[-1,1].
  c3  3D 25-point star, R=4, 8th-order central second-difference weights on each axis
      normalised to sum|w| = 1; 512^3 fp32; ZERO; 4 steps; input = 0.99 x mean of 8
      random-phase sinusoids + 0.01 x U[-1,1] noise.
  c4  3D 27-point box, R=1, 27 i.i.d. U[-1,1] weights normalised to sum|w| = 1 (fp64, then
      rounded to fp32), coefficient field k i.i.d. U[0.5,1]; 512^3 fp32; PERIODIC; 1 step;
      input i.i.d. U[-1,1].
  c5  depthwise 3x3x3 in convolution form: N=8, C=32, 128^3 fp32; per-channel weights
      i.i.d. U[-1,1] normalised per channel; ZERO (padding 1); 1 step; input i.i.d. N(0,1).
  c5b the same recipe in fp64 at N=2 (separate draws).
  paper  the paper's own case: 2D box R=3 (49 points), 10240^2 fp64, ZERO (padding 3);
      weights not printed in the paper, so i.i.d. U[-1,1] normalised to sum|w| = 1.
  c2_512  the c2 recipe on 512^3 (a working set beyond the Infinity Cache, where four
      steps per pass pay off); context for the temporal-depth rule, not one of the five.
"""
from __future__ import annotations

from dataclasses import dataclass, replace
from fractions import Fraction

import numpy as np

STAR, BOX = 0, 1
ZERO, PERIODIC = 0, 1


@dataclass(frozen=True)
class Workload:
    name: str
    ndim: int
    dims: tuple            # (nz, ny, nx) or (ny, nx)
    batch: int             # N*C volumes for the conv form, else 1
    channels: int          # weight sets; volume b uses set b % channels
    dtype: str             # "f32" or "f64"
    shape: int             # STAR or BOX
    radius: int
    boundary: int          # ZERO or PERIODIC
    steps: int
    has_field: bool
    seed: int
    recipe: str            # input recipe tag
    n: int = 1             # conv-form N (batch = n * channels)

    @property
    def npoints(self) -> int:
        side = 2 * self.radius + 1
        return 1 + 2 * self.ndim * self.radius if self.shape == STAR else side ** self.ndim

    @property
    def points_per_step(self) -> int:
        return int(np.prod(self.dims)) * self.batch

    @property
    def itemsize(self) -> int:
        return 4 if self.dtype == "f32" else 8

    @property
    def np_dtype(self):
        return np.float32 if self.dtype == "f32" else np.float64

    def resized(self, dims, n: int | None = None, steps: int | None = None) -> "Workload":
        """The same recipe on other extents (and batch N, steps) for reduced-size tests."""
        n = self.n if n is None else n
        return replace(self, dims=tuple(int(d) for d in dims), n=n,
                       batch=n * self.channels if self.recipe == "conv" else self.batch,
                       steps=self.steps if steps is None else steps)


WORKLOADS = {
    "c1": Workload("c1", 2, (256, 256), 1, 1, "f32", STAR, 1, ZERO, 1, False, 1, "laplace2d"),
    "c2": Workload("c2", 3, (256, 256, 256), 1, 1, "f32", STAR, 1, ZERO, 10, False, 2,
                   "star7"),
    "c3": Workload("c3", 3, (512, 512, 512), 1, 1, "f32", STAR, 4, ZERO, 4, False, 3,
                   "fd8"),
    "c4": Workload("c4", 3, (512, 512, 512), 1, 1, "f32", BOX, 1, PERIODIC, 1, True, 4,
                   "box_field"),
    "c5": Workload("c5", 3, (128, 128, 128), 8 * 32, 32, "f32", BOX, 1, ZERO, 1, False, 5,
                   "conv", n=8),
    "c5b": Workload("c5b", 3, (128, 128, 128), 2 * 32, 32, "f64", BOX, 1, ZERO, 1, False, 6,
                    "conv", n=2),
    "paper": Workload("paper", 2, (10240, 10240), 1, 1, "f64", BOX, 3, ZERO, 10240, False, 7,
                      "box_uniform"),
    "c2_512": Workload("c2_512", 3, (512, 512, 512), 1, 1, "f32", STAR, 1, ZERO, 10, False, 2,
                       "star7"),
}


def fd8_second_derivative() -> list:
    """Exact 8th-order central second-difference weights c_0..c_4 (offsets 0..4)."""
    return [Fraction(-205, 72), Fraction(8, 5), Fraction(-1, 5), Fraction(8, 315),
            Fraction(-1, 560)]


def fd8_star_weights_exact(ndim: int = 3) -> list:
    """25-point (3D) star weights as exact rationals, in star order (centre, then per axis
    -4..-1, +1..+4), normalised so that the sum of absolute values is 1."""
    c = fd8_second_derivative()
    raw = [ndim * c[0]]
    for _axis in range(ndim):
        raw += [c[4], c[3], c[2], c[1], c[1], c[2], c[3], c[4]]
    s = sum(abs(v) for v in raw)
    return [v / s for v in raw]


def _uniform(rng, size, lo, hi, dtype):
    """i.i.d. U[lo, hi) in the requested dtype, drawn as float64 and rounded."""
    return rng.uniform(lo, hi, size=size).astype(dtype)


def _normalised(rng, count, channels):
    """channels x count i.i.d. U[-1,1] weights, each row scaled to sum|w| = 1 (fp64)."""
    raw = rng.uniform(-1.0, 1.0, size=(channels, count))
    return raw / np.abs(raw).sum(axis=1, keepdims=True)


def _sinusoids(rng, dims):
    """0.99 * (1/8) * sum_m sin(2 pi k_m . p / n + phi_m), k_m in {0..8}^3 minus 0, in fp64.
    Evaluated plane by plane with sin(a + b) = sin a cos b + cos a sin b, a = phase along x,
    b = phase along (z, y)."""
    nz, ny, nx = dims
    ks = []
    while len(ks) < 8:
        k = tuple(int(v) for v in rng.integers(0, 9, size=3))
        if k != (0, 0, 0):
            ks.append(k)
    phis = rng.uniform(0.0, 2.0 * np.pi, size=8)
    out = np.zeros(dims, dtype=np.float64)
    z = np.arange(nz)[:, None]
    y = np.arange(ny)[None, :]
    x = np.arange(nx)
    for (kz, ky, kx), phi in zip(ks, phis):
        a = 2.0 * np.pi * kx * x / nx + phi                 # (nx,)
        b = 2.0 * np.pi * (kz * z / nz + ky * y / ny)       # (nz, ny)
        sa, ca, sb, cb = np.sin(a), np.cos(a), np.sin(b), np.cos(b)
        for zi in range(nz):
            out[zi] += sb[zi][:, None] * ca[None, :] + cb[zi][:, None] * sa[None, :]
    return out * (0.99 / 8.0)


def make(w: Workload):
    """Return (x, weights, field) for a workload.

    x: (*dims) for batch 1, (N, C, *dims) for the conv form; dtype per workload.
    weights: (channels, npoints), same dtype.  field: x-shaped or None.
    """
    rng = np.random.Generator(np.random.PCG64(w.seed))
    dt = w.np_dtype
    field = None
    if w.recipe == "laplace2d":
        x = _uniform(rng, w.dims, -1.0, 1.0, dt)
        wts = np.array([[-1.0, 0.25, 0.25, 0.25, 0.25]])
    elif w.recipe == "star7":
        x = _uniform(rng, w.dims, -1.0, 1.0, dt)
        wts = np.array([[0.4] + [0.1] * 6])
    elif w.recipe == "fd8":
        if w.ndim != 3:
            raise ValueError("fd8 recipe is 3D")
        sig = _sinusoids(rng, w.dims)
        noise = rng.uniform(-1.0, 1.0, size=w.dims)
        x = (sig + 0.01 * noise).astype(dt)
        wts = np.array([[float(v) for v in fd8_star_weights_exact(3)]])
    elif w.recipe == "box_field":
        x = _uniform(rng, w.dims, -1.0, 1.0, dt)
        wts = _normalised(rng, w.npoints, w.channels)
        field = _uniform(rng, w.dims, 0.5, 1.0, dt)
    elif w.recipe == "conv":
        shp = (w.n, w.channels) + tuple(w.dims)
        x = rng.standard_normal(size=shp, dtype=dt)
        wts = _normalised(rng, w.npoints, w.channels)
    elif w.recipe == "box_uniform":
        x = _uniform(rng, w.dims, -1.0, 1.0, dt)
        wts = _normalised(rng, w.npoints, w.channels)
    else:
        raise ValueError("unknown recipe %r" % w.recipe)
    return x, np.ascontiguousarray(wts.astype(dt)), field
