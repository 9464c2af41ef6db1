"""The piecewise whole-grid oracle (``oracle/whole_grid.py``) against the whole-grid
oracle: every kept point must be bit-identical, for both boundaries, 2D and 3D, batches
with several weight sets, a coefficient field, step counts whose reach exceeds a slab,
and slab counts that cut the grid into pieces thinner than their halo.  ``compare`` must
find a planted error at its place and count non-finite values."""
import numpy as np
import pytest

import oracle
from oracle import whole_grid

STAR, BOX = oracle.STAR, oracle.BOX
ZERO, PERIODIC = oracle.ZERO, oracle.PERIODIC


def _case(seed, dims, *, shape, radius, ndim, batch=1, channels=1, field=False):
    g = np.random.default_rng(seed)
    lead = (batch,) if batch > 1 else ()
    x = g.uniform(-1, 1, lead + tuple(dims))
    npts = oracle.num_points(shape, ndim, radius)
    w = g.uniform(-1, 1, (channels, npts))
    w /= np.abs(w).sum(axis=1, keepdims=True)
    k = g.uniform(0.5, 1.0, x.shape) if field else None
    return x, w, k


CASES = [
    # (dims, shape, radius, ndim, batch, channels, field)
    ((23, 9, 11), STAR, 2, 3, 1, 1, False),
    ((31, 7, 8), BOX, 1, 3, 1, 1, True),
    ((17, 6, 5), STAR, 4, 3, 1, 1, False),
    ((40, 13), BOX, 3, 2, 1, 1, False),
    ((29, 10), STAR, 1, 2, 1, 1, False),
    ((9, 5, 6), BOX, 1, 3, 4, 2, True),
]


@pytest.mark.parametrize("boundary", [ZERO, PERIODIC])
@pytest.mark.parametrize("steps", [0, 1, 2, 3])
@pytest.mark.parametrize("count", [None, 2, 5, 11])
@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c[0])))
def test_pieces_equal_whole_grid(case, count, steps, boundary):
    dims, shape, radius, ndim, batch, channels, field = case
    x, w, k = _case(7, dims, shape=shape, radius=radius, ndim=ndim, batch=batch,
                    channels=channels, field=field)
    kw = dict(shape=shape, radius=radius, boundary=boundary, steps=steps, ndim=ndim,
              channels=channels, field=k)
    whole = oracle.apply(x, w, **kw)
    pieced = whole_grid.evaluate(x, w, threads=3, count=count, **kw)
    assert np.array_equal(whole, pieced)


def test_pieces_cover_every_plane_once():
    x = np.zeros((50, 4, 4))
    for boundary in (ZERO, PERIODIC):
        for count in (1, 3, 7, 50):
            pcs = whole_grid.pieces(x, radius=2, boundary=boundary, steps=2, ndim=3,
                                    count=count)
            seen = np.zeros(50, dtype=int)
            for pc in pcs:
                seen[pc["dst"]] += 1
                kept = (pc["keep"].stop - pc["keep"].start)
                assert kept == pc["dst"].stop - pc["dst"].start
            assert (seen == 1).all()


def test_compare_finds_a_planted_error_and_nans():
    dims = (21, 8, 9)
    x, w, k = _case(3, dims, shape=STAR, radius=2, ndim=3)
    kw = dict(shape=STAR, radius=2, boundary=ZERO, steps=2, ndim=3)
    ref = oracle.apply(x, w, **kw)
    rep = whole_grid.compare(ref.astype(np.float32), x, w, threads=2, count=4, **kw)
    assert rep["points"] == x.size and rep["nonfinite"] == 0
    assert rep["max_abs_err"] < 1e-6
    bad = ref.copy()
    flat = np.ravel_multi_index((11, 3, 4), dims)   # a plane next to a slab cut
    bad.flat[flat] += 1e-3
    rep = whole_grid.compare(bad, x, w, threads=2, count=4, **kw)
    assert rep["worst"] == flat and abs(rep["max_abs_err"] - 1e-3) < 1e-12
    bad.flat[5] = np.nan
    rep = whole_grid.compare(bad, x, w, threads=2, count=4, **kw)
    assert rep["nonfinite"] == 1 and rep["max_abs_err"] == np.inf


def test_compare_batch_locates_the_volume():
    x, w, k = _case(5, (6, 5, 8), shape=BOX, radius=1, ndim=3, batch=6, channels=3,
                    field=True)
    kw = dict(shape=BOX, radius=1, boundary=ZERO, steps=1, ndim=3, channels=3, field=k)
    ref = oracle.apply(x, w, **kw)
    bad = ref.copy()
    bad[4, 2, 1, 7] -= 2e-4
    rep = whole_grid.compare(bad, x, w, threads=2, **kw)
    assert rep["worst"] == np.ravel_multi_index((4, 2, 1, 7), x.shape)
    assert rep["pieces"] == 6 and rep["points"] == x.size
