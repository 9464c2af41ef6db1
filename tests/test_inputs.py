"""Seeded workload generators: reproducibility, ranges, and the 8th-order weights."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from paper_2608_21157_amd import inputs
from paper_2608_21157_amd.inputs import WORKLOADS, fd8_second_derivative, fd8_star_weights_exact

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_fd8_weights_are_exact_on_polynomials_to_degree_9():
    """sum_r c_|r| r^m = m! * [m == 2]  for m = 0..9  (odd m vanish by symmetry)."""
    c = fd8_second_derivative()
    for m in range(10):
        s = sum(c[abs(r)] * Fraction(r) ** m for r in range(-4, 5))
        assert s == (2 if m == 2 else 0), m
    # not exact at degree 10: the truncation term
    assert sum(c[abs(r)] * Fraction(r) ** 10 for r in range(-4, 5)) != 0


def test_fd8_weights_match_golden_table():
    with open(os.path.join(GOLDEN, "fd8_weights.json")) as f:
        gold = json.load(f)
    assert [Fraction(v) for v in gold["c"]] == fd8_second_derivative()
    wx = fd8_star_weights_exact(3)
    assert sum(abs(v) for v in wx) == 1
    S = 3 * abs(fd8_second_derivative()[0]) + 6 * sum(abs(v) for v in fd8_second_derivative()[1:])
    assert S == Fraction(gold["sum_abs_3d_raw"])
    n = gold["normalised_3d"]
    assert wx[0] == Fraction(n["centre"])
    # star order: per axis -4, -3, -2, -1, +1, +2, +3, +4
    for axis in range(3):
        seg = wx[1 + 8 * axis: 9 + 8 * axis]
        assert seg == [Fraction(n[k]) for k in ("4", "3", "2", "1", "1", "2", "3", "4")]


def test_c3_fp32_weights_are_exact():
    """All normalised c3 weights but +-3 (1/768) are dyadic and exact in fp32."""
    _, w, _ = inputs.make(WORKLOADS["c3"].resized((16, 16, 16)))
    exact = [float(v) for v in fd8_star_weights_exact(3)]
    assert w.dtype == np.float32 and w.shape == (1, 25)
    for a, b in zip(w[0], exact):
        if abs(b) != 1 / 768:
            assert float(a) == b


def test_paper_case_matches_golden():
    with open(os.path.join(GOLDEN, "paper_case_study.json")) as f:
        gold = json.load(f)
    w = WORKLOADS["paper"]
    assert w.ndim == gold["ndim"] and w.radius == gold["radius"]
    assert tuple(w.dims) == tuple(gold["grid"]) and w.steps == gold["steps"]
    assert w.npoints == gold["points"] and w.dtype == gold["precision"].replace("fp", "f")
    assert w.boundary == inputs.ZERO and w.shape == inputs.BOX


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5", "c5b", "paper", "c2_512"])
def test_reduced_workloads_are_seeded_and_in_range(name):
    base = WORKLOADS[name]
    dims = (12, 10) if base.ndim == 2 else (6, 10, 12)
    wl = base.resized(dims, n=2 if base.recipe == "conv" else None)
    x1, w1, k1 = inputs.make(wl)
    x2, w2, k2 = inputs.make(wl)
    assert np.array_equal(x1, x2) and np.array_equal(w1, w2)
    assert x1.dtype == wl.np_dtype and w1.dtype == wl.np_dtype
    assert w1.shape == (wl.channels, wl.npoints)
    if wl.recipe == "conv":
        assert x1.shape == (2, wl.channels) + dims
    else:
        assert x1.shape == dims
    if wl.recipe != "conv":
        assert np.abs(x1).max() <= 1.0
    if wl.recipe in ("box_field", "conv", "box_uniform"):
        np.testing.assert_allclose(np.abs(w1.astype(np.float64)).sum(axis=1), 1.0, rtol=1e-6)
    if wl.has_field:
        assert k1 is not None and k1.min() >= 0.5 and k1.max() <= 1.0
        assert np.array_equal(k1, k2)
    else:
        assert k1 is None


def test_fixed_weights():
    _, w, _ = inputs.make(WORKLOADS["c1"].resized((4, 4)))
    assert w.tolist() == [[-1.0, 0.25, 0.25, 0.25, 0.25]]
    _, w, _ = inputs.make(WORKLOADS["c2"].resized((4, 4, 4)))
    np.testing.assert_array_equal(w, np.array([[0.4] + [0.1] * 6], np.float32))


def test_sinusoid_recipe_is_bounded_and_not_constant():
    x, _, _ = inputs.make(WORKLOADS["c3"].resized((16, 16, 16)))
    assert np.abs(x).max() <= 1.0
    assert x.std() > 0.05


def test_full_size_shapes_declared():
    assert WORKLOADS["c3"].points_per_step == 512 ** 3
    assert WORKLOADS["c5"].points_per_step == 8 * 32 * 128 ** 3
    assert WORKLOADS["c5b"].points_per_step == 2 * 32 * 128 ** 3
    assert WORKLOADS["c4"].has_field and WORKLOADS["c4"].boundary == inputs.PERIODIC
