"""Plausible mistakes planted in a copy of the oracle must fail at least one pin.

Each mutant is ``oracle.c`` with one textual change (a sign, an axis, a dropped term, a
wrong wrap, a wrong channel, an off-by-one step count, a reordered offset table), compiled
on the CPU into a temporary directory and run through a compact battery of the pins in
``test_oracle.py``.  The unmodified source must pass every check.
"""
import os

import numpy as np
import pytest
import scipy.ndimage as ndi
import torch

import oracle
from oracle import BOX, PERIODIC, STAR, ZERO

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")

MUTANTS = {
    "x_offset_sign": ("x + off[3 * j + 2]);", "x - off[3 * j + 2]);"),
    "y_reads_x_offset": ("y + off[3 * j + 1], x + off[3 * j + 2]);",
                         "y + off[3 * j + 2], x + off[3 * j + 2]);"),
    "dropped_first_term": ("for (int j = 0; j < npts; ++j) {\n                            const double v = read_bnd",
                           "for (int j = 1; j < npts; ++j) {\n                            const double v = read_bnd"),
    "zero_acts_periodic": ("if (boundary == ORACLE_ZERO) {\n        if (z < 0",
                           "if (boundary == -1) {\n        if (z < 0"),
    "wrap_clamps": ("return (m < 0) ? m + n : m;", "return (m < 0) ? 0 : m;"),
    "channel_by_division": ("const double *wb = w + (size_t)(b % channels) * (size_t)npts;\n        const double *kb = field ? field + b * vol : NULL;\n        memcpy",
                            "const double *wb = w + (size_t)(b / channels % channels) * (size_t)npts;\n        const double *kb = field ? field + b * vol : NULL;\n        memcpy"),
    "field_dropped": ("acc += kb[p] * wb[j] * v;", "acc += wb[j] * v;"),
    "one_step_short": ("for (int s = 0; s < steps; ++s)", "for (int s = 1; s < steps; ++s)"),
    "star_axis_reversed": ("for (int r = -radius; r <= radius; ++r) {",
                           "for (int r = radius; r >= -radius; --r) {"),
    "box_yx_transposed": ("off[3 * j + 1] = oy;\n                    off[3 * j + 2] = ox;",
                          "off[3 * j + 1] = ox;\n                    off[3 * j + 2] = oy;"),
}


def _close(a, b, tol=1e-12):
    return a.shape == b.shape and np.allclose(a, b, rtol=0, atol=tol)


def battery(lib):
    """Return the names of the failed checks."""
    g = np.random.default_rng(5)
    failed = []
    # zero box, non-cubic, asymmetric weights, 2 steps, vs scipy
    x = g.uniform(-1, 1, (5, 6, 7))
    w = g.uniform(-1, 1, 27)
    K = w.reshape(3, 3, 3)
    got = oracle.apply(x, w, shape=BOX, radius=1, boundary=ZERO, steps=2, lib=lib)
    if not _close(got, ndi.correlate(ndi.correlate(x, K, mode="constant"), K, mode="constant")):
        failed.append("scipy_box_zero")
    # periodic star R=2 vs roll
    off = [(0, 0, 0)] + [(r, 0, 0) for r in (-2, -1, 1, 2)] + [(0, r, 0) for r in (-2, -1, 1, 2)] \
        + [(0, 0, r) for r in (-2, -1, 1, 2)]
    ws = g.uniform(-1, 1, 13)
    got = oracle.apply(x, ws, shape=STAR, radius=2, boundary=PERIODIC, steps=1, lib=lib)
    ref = sum(wj * np.roll(x, (-o[0], -o[1], -o[2]), (0, 1, 2)) for wj, o in zip(ws, off))
    if not _close(got, ref):
        failed.append("roll_star_periodic")
    # depthwise conv form vs torch, N=2, C=3
    xc = g.standard_normal((2, 3, 4, 5, 6))
    wc = g.uniform(-1, 1, (3, 27))
    got = oracle.apply(xc, wc, shape=BOX, radius=1, boundary=ZERO, channels=3, lib=lib)
    ref = torch.nn.functional.conv3d(torch.from_numpy(xc), torch.from_numpy(wc).reshape(3, 1, 3, 3, 3),
                                     padding=1, groups=3).numpy()
    if not _close(got, ref):
        failed.append("torch_depthwise")
    # output-indexed field, periodic
    k = g.uniform(0.5, 1, x.shape)
    got = oracle.apply(x, w, shape=BOX, radius=1, boundary=PERIODIC, field=k, lib=lib)
    if not _close(got, k * ndi.correlate(x, K, mode="wrap")):
        failed.append("field_periodic")
    # steps=3 vs scipy for a 2D R=1 star
    x2 = g.uniform(-1, 1, (7, 9))
    w2 = g.uniform(-1, 1, 5)
    K2 = np.zeros((3, 3))
    K2[1, 1], K2[0, 1], K2[2, 1], K2[1, 0], K2[1, 2] = w2
    ref = x2
    for _ in range(3):
        ref = ndi.correlate(ref, K2, mode="constant")
    got = oracle.apply(x2, w2, shape=STAR, radius=1, boundary=ZERO, steps=3, ndim=2, lib=lib)
    if not _close(got, ref):
        failed.append("scipy_star2d_3steps")
    return failed


def test_unmutated_oracle_passes_battery(oracle_lib):
    assert battery(None) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, "mutation anchor not found: %s" % name
    mutated = src.replace(old, new, 1)
    path = tmp_path / ("oracle_%s.c" % name)
    path.write_text(mutated)
    lib = oracle.bind(oracle.compile_source(str(path), str(tmp_path / ("lib_%s.so" % name))))
    assert battery(lib), "mutant %s passed every check" % name
