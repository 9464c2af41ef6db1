"""Pins for the fp64 CPU oracle: it is checked against things other than itself.

Each test ties the oracle to the operator's definition (HIERA, experimental setup,
"Case-study protocol": zero-padded cross-correlation, padding R, stride 1, iterated, FP64)
through an independent route: library routines (scipy.ndimage.correlate, torch conv in
fp64 on the CPU, numpy.roll), closed forms (constants, quadratics, polynomials that the
8th-order stencil differentiates exactly), eigenfunctions (periodic plane waves, Dirichlet
sine modes), invariants (composition, translation, reflection, linearity, norm bound) and a
dense operator matrix built pair by pair on tiny grids.  ``test_oracle_mutants.py`` shows
that plausible mistakes in the oracle fail these pins.
"""
import itertools

import numpy as np
import pytest
import scipy.ndimage as ndi
import torch

import oracle
from oracle import BOX, PERIODIC, STAR, ZERO


def rng(seed=0):
    return np.random.default_rng(seed)


def star_to_box(wstar, ndim, R):
    """Embed star weights (oracle order) into a (2R+1)^ndim correlation kernel."""
    K = np.zeros((2 * R + 1,) * ndim)
    c = (R,) * ndim
    K[c] = wstar[0]
    j = 1
    for axis in range(ndim):
        for r in list(range(-R, 0)) + list(range(1, R + 1)):
            idx = list(c)
            idx[axis] += r
            K[tuple(idx)] = wstar[j]
            j += 1
    return K


def box_kernel(wbox, ndim, R):
    return np.asarray(wbox, dtype=np.float64).reshape((2 * R + 1,) * ndim)


# ----------------------------------------------------------------------------- offsets

def test_point_counts():
    for ndim in (2, 3):
        for R in range(0, 5):
            assert oracle.num_points(STAR, ndim, R) == 1 + 2 * ndim * R
            assert oracle.num_points(BOX, ndim, R) == (2 * R + 1) ** ndim
    # the paper's case: radius 3, 7x7 = 49 points
    assert oracle.num_points(BOX, 2, 3) == 49
    assert oracle.num_points(BOX, 4, 1) == -1
    assert oracle.num_points(7, 3, 1) == -1


def test_offset_order_box_is_lexicographic():
    for ndim, R in [(2, 1), (2, 3), (3, 1), (3, 2)]:
        off = oracle.offsets(BOX, ndim, R)
        rngs = [range(-R, R + 1)] * ndim
        expect = [((0,) if ndim == 2 else ()) + t for t in itertools.product(*rngs)]
        assert [tuple(o) for o in off] == expect


def test_offset_order_star():
    off = oracle.offsets(STAR, 3, 2)
    assert tuple(off[0]) == (0, 0, 0)
    assert [tuple(o) for o in off[1:5]] == [(-2, 0, 0), (-1, 0, 0), (1, 0, 0), (2, 0, 0)]
    assert [tuple(o) for o in off[5:9]] == [(0, -2, 0), (0, -1, 0), (0, 1, 0), (0, 2, 0)]
    assert [tuple(o) for o in off[9:13]] == [(0, 0, -2), (0, 0, -1), (0, 0, 1), (0, 0, 2)]
    off2 = oracle.offsets(STAR, 2, 1)
    assert [tuple(o) for o in off2] == [(0, 0, 0), (0, -1, 0), (0, 1, 0), (0, 0, -1), (0, 0, 1)]


# ----------------------------------------------------------------------------- libraries

def scipy_steps(x, K, steps, mode):
    for _ in range(steps):
        x = ndi.correlate(x, K, mode=mode, cval=0.0)
    return x


@pytest.mark.parametrize("ndim,dims", [(2, (9, 11)), (3, (5, 6, 7)), (3, (7, 4, 9))])
@pytest.mark.parametrize("R", [1, 2, 3])
@pytest.mark.parametrize("steps", [1, 2, 3])
def test_box_zero_matches_scipy(ndim, dims, R, steps):
    g = rng(100 + R + 10 * steps)
    x = g.uniform(-1, 1, dims)
    w = g.uniform(-1, 1, (2 * R + 1) ** ndim)
    got = oracle.apply(x, w, shape=BOX, radius=R, boundary=ZERO, steps=steps, ndim=ndim)
    ref = scipy_steps(x, box_kernel(w, ndim, R), steps, "constant")
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("ndim,dims", [(2, (9, 11)), (3, (6, 5, 13))])
@pytest.mark.parametrize("R", [1, 2, 4])
@pytest.mark.parametrize("boundary,mode", [(ZERO, "constant"), (PERIODIC, "wrap")])
def test_star_matches_scipy(ndim, dims, R, boundary, mode):
    g = rng(200 + R)
    x = g.uniform(-1, 1, dims)
    w = g.uniform(-1, 1, 1 + 2 * ndim * R)
    got = oracle.apply(x, w, shape=STAR, radius=R, boundary=boundary, steps=2, ndim=ndim)
    ref = scipy_steps(x, star_to_box(w, ndim, R), 2, mode)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_zero_matches_torch_conv_depthwise():
    """Conv form: N=2, C=3 volumes, volume b = n*C + c uses weight set c (torch groups=C)."""
    g = rng(7)
    N, C, D, H, W = 2, 3, 5, 6, 7
    x = g.standard_normal((N, C, D, H, W))
    w = g.uniform(-1, 1, (C, 27))
    got = oracle.apply(x, w, shape=BOX, radius=1, boundary=ZERO, steps=1, ndim=3, channels=C)
    ref = torch.nn.functional.conv3d(torch.from_numpy(x), torch.from_numpy(w).reshape(C, 1, 3, 3, 3),
                                     padding=1, groups=C).numpy()
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_zero_matches_torch_conv2d_paper_case():
    """The paper's operator: single-channel 7x7 zero-padded cross-correlation, pad 3, FP64."""
    g = rng(8)
    x = g.uniform(-1, 1, (23, 17))
    w = g.uniform(-1, 1, 49)
    got = oracle.apply(x, w, shape=BOX, radius=3, boundary=ZERO, steps=3, ndim=2)
    t = torch.from_numpy(x)[None, None]
    K = torch.from_numpy(w).reshape(1, 1, 7, 7)
    for _ in range(3):
        t = torch.nn.functional.conv2d(t, K, padding=3)
    np.testing.assert_allclose(got, t[0, 0].numpy(), rtol=0, atol=1e-12)


@pytest.mark.parametrize("dims", [(1, 1, 1), (2, 3, 1), (3, 2, 2), (4, 5, 6)])
@pytest.mark.parametrize("shape,R", [(BOX, 1), (BOX, 2), (STAR, 3), (STAR, 4)])
def test_periodic_matches_roll_tiny(dims, shape, R):
    """Periodic = sum_o w_o * roll(x, -o); extents smaller than R wrap several times."""
    g = rng(9)
    x = g.uniform(-1, 1, dims)
    off = oracle.offsets(shape, 3, R)
    w = g.uniform(-1, 1, len(off))
    got = oracle.apply(x, w, shape=shape, radius=R, boundary=PERIODIC, steps=2, ndim=3)
    u = x
    for _ in range(2):
        u = sum(wj * np.roll(u, shift=(-o[0], -o[1], -o[2]), axis=(0, 1, 2)) for wj, o in zip(w, off))
    np.testing.assert_allclose(got, u, rtol=0, atol=1e-12)


def test_zero_tiny_extents_read_zero():
    """Extents below 2R+1: everything beyond the grid reads as zero."""
    g = rng(10)
    for dims in [(1, 1, 1), (1, 2, 3), (2, 1, 1)]:
        x = g.uniform(-1, 1, dims)
        w = g.uniform(-1, 1, 7 ** 3)
        got = oracle.apply(x, w, shape=BOX, radius=3, boundary=ZERO, steps=2, ndim=3)
        ref = scipy_steps(x, box_kernel(w, 3, 3), 2, "constant")
        np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("boundary,mode", [(ZERO, "constant"), (PERIODIC, "wrap")])
def test_field_is_indexed_by_output_point(boundary, mode):
    g = rng(11)
    x = g.uniform(-1, 1, (6, 7, 8))
    w = g.uniform(-1, 1, 27)
    k = g.uniform(0.5, 1.0, x.shape)
    got = oracle.apply(x, w, shape=BOX, radius=1, boundary=boundary, steps=2, field=k)
    u = x
    for _ in range(2):
        u = k * ndi.correlate(u, box_kernel(w, 3, 1), mode=mode)
    np.testing.assert_allclose(got, u, rtol=0, atol=1e-12)


def test_batch_channels_periodic_field():
    g = rng(12)
    N, C = 2, 3
    x = g.uniform(-1, 1, (N, C, 4, 5, 6))
    w = g.uniform(-1, 1, (C, 27))
    k = g.uniform(0.5, 1, x.shape)
    got = oracle.apply(x, w, shape=BOX, radius=1, boundary=PERIODIC, steps=1, field=k, channels=C)
    for n in range(N):
        for c in range(C):
            ref = k[n, c] * ndi.correlate(x[n, c], box_kernel(w[c], 3, 1), mode="wrap")
            np.testing.assert_allclose(got[n, c], ref, rtol=0, atol=1e-12)


# ----------------------------------------------------------------------------- closed forms

def test_constant_field():
    g = rng(13)
    c = 0.7
    for shape, R in [(STAR, 1), (STAR, 4), (BOX, 1)]:
        n = oracle.num_points(shape, 3, R)
        w = g.uniform(-1, 1, n)
        x = np.full((2 * R + 3,) * 3, c)
        z = oracle.apply(x, w, shape=shape, radius=R, boundary=ZERO, steps=1)
        inner = z[R:-R, R:-R, R:-R]
        np.testing.assert_allclose(inner, c * w.sum(), rtol=1e-14, atol=1e-15)
        k = g.uniform(0.5, 1, x.shape)
        p = oracle.apply(x, w, shape=shape, radius=R, boundary=PERIODIC, steps=1, field=k)
        np.testing.assert_allclose(p, k * c * w.sum(), rtol=1e-13, atol=1e-15)
    # the 5-point Laplacian of a constant is 0, the 7-point c2 star keeps it
    x = np.full((6, 6), 3.0)
    z = oracle.apply(x, [-1, .25, .25, .25, .25], shape=STAR, radius=1, ndim=2)
    assert np.all(z[1:-1, 1:-1] == 0.0)


def test_quadratic_laplace2d_exact():
    """0.25 * discrete Laplacian of a x^2 + b y^2 + c xy + d x + e y + g is 0.5 (a + b),
    exactly (dyadic coefficients, small integers)."""
    a, b, c, d, e, g0 = 3.0, -1.5, 2.0, 0.5, -4.0, 7.0
    y, x = np.meshgrid(np.arange(-8, 9, dtype=float), np.arange(-7, 8, dtype=float), indexing="ij")
    f = a * x * x + b * y * y + c * x * y + d * x + e * y + g0
    z = oracle.apply(f, [-1, .25, .25, .25, .25], shape=STAR, radius=1, ndim=2)
    assert np.all(z[1:-1, 1:-1] == 0.5 * (a + b))


def test_quadratic_star7():
    """I + 0.1 * Laplacian on a 3D quadratic: f + 0.2 (a + b + c) in the interior."""
    a, b, c = 0.25, -0.5, 1.0
    z, y, x = np.meshgrid(*(np.arange(-4, 5, dtype=float),) * 3, indexing="ij")
    f = a * x * x + b * y * y + c * z * z + 0.5 * x * y - z + 2.0
    out = oracle.apply(f, [0.4] + [0.1] * 6, shape=STAR, radius=1)
    np.testing.assert_allclose(out[1:-1, 1:-1, 1:-1], (f + 0.2 * (a + b + c))[1:-1, 1:-1, 1:-1],
                               rtol=1e-13, atol=1e-13)


FD8_INT = [-14350, 8064, -1008, 128, -9]   # 5040 * (-205/72, 8/5, -1/5, 8/315, -1/560)


def fd8_star_int(ndim):
    c = FD8_INT
    return [ndim * c[0]] + [c[4], c[3], c[2], c[1], c[1], c[2], c[3], c[4]] * ndim


def test_fd8_differentiates_x8_exactly():
    """The 8th-order stencil is exact on degree <= 9: one step on x^8 gives 5040*56*x^6
    (bit-exact: all intermediates are integers below 2^53)."""
    r = np.arange(-16, 17, dtype=float)
    Z, Y, X = np.meshgrid(r, r, r, indexing="ij")
    out = oracle.apply(X ** 8, fd8_star_int(3), shape=STAR, radius=4, boundary=ZERO, steps=1)
    s = slice(4, -4)
    assert np.array_equal(out[s, s, s], (5040 * 56 * X ** 6)[s, s, s])
    # the axis of differentiation matters: the same field along z
    out = oracle.apply(Z ** 8, fd8_star_int(3), shape=STAR, radius=4, boundary=ZERO, steps=1)
    assert np.array_equal(out[s, s, s], (5040 * 56 * Z ** 6)[s, s, s])


def test_fd8_two_steps_on_x4():
    """Two steps on x^4: d^2 x^4 = 12 x^2, d^2 12 x^2 = 24, times 5040^2 = 609,638,400."""
    r = np.arange(-16, 17, dtype=float)
    Z, Y, X = np.meshgrid(r, r, r, indexing="ij")
    out = oracle.apply(Y ** 4, fd8_star_int(3), shape=STAR, radius=4, boundary=ZERO, steps=2)
    s = slice(8, -8)
    assert np.all(out[s, s, s] == 609_638_400.0)


# ----------------------------------------------------------------------------- eigenfunctions

@pytest.mark.parametrize("shape,R", [(BOX, 1), (STAR, 4), (STAR, 1), (BOX, 2)])
@pytest.mark.parametrize("steps", [1, 3])
def test_periodic_plane_wave(shape, R, steps):
    """cos(theta.p) -> Re(lam^s e^{i theta.p}) with lam = sum_o w_o e^{i theta.o}: the sign
    of the offsets (correlation, not convolution) decides Im(lam) for asymmetric w."""
    g = rng(14)
    dims = (8, 10, 12)
    m = (1, 3, 2)
    off = oracle.offsets(shape, 3, R)
    w = g.uniform(-1, 1, len(off))
    w /= np.abs(w).sum()
    theta = 2 * np.pi * np.array(m) / np.array(dims)
    lam = np.sum(w * np.exp(1j * (off @ theta)))
    P = np.stack(np.meshgrid(*[np.arange(n) for n in dims], indexing="ij"), -1)
    ph = P @ theta
    x = np.cos(ph)
    got = oracle.apply(x, w, shape=shape, radius=R, boundary=PERIODIC, steps=steps)
    ref = np.real(lam ** steps * np.exp(1j * ph))
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_dirichlet_sine_modes_star7_ten_steps():
    """Zero boundary, symmetric R=1 star: prod sin(pi m_a (p_a+1)/(n_a+1)) is an eigenvector
    with lam = w0 + sum_a 2 w1 cos(pi m_a/(n_a+1)); ten steps scale it by lam^10."""
    dims = (9, 10, 11)
    m = (2, 1, 5)
    grids = np.meshgrid(*[np.arange(n) for n in dims], indexing="ij")
    x = np.ones(dims)
    lam = 0.4
    for a in range(3):
        x = x * np.sin(np.pi * m[a] * (grids[a] + 1) / (dims[a] + 1))
        lam += 2 * 0.1 * np.cos(np.pi * m[a] / (dims[a] + 1))
    got = oracle.apply(x, [0.4] + [0.1] * 6, shape=STAR, radius=1, boundary=ZERO, steps=10)
    np.testing.assert_allclose(got, lam ** 10 * x, rtol=0, atol=1e-13)


# ----------------------------------------------------------------------------- invariants

def test_composition_bit_exact():
    g = rng(15)
    x = g.uniform(-1, 1, (6, 7, 8))
    w = g.uniform(-1, 1, 25)
    for boundary in (ZERO, PERIODIC):
        one = x
        for _ in range(3):
            one = oracle.apply(one, w, shape=STAR, radius=4, boundary=boundary, steps=1)
        three = oracle.apply(x, w, shape=STAR, radius=4, boundary=boundary, steps=3)
        assert np.array_equal(one, three)
    zero = oracle.apply(x, w, shape=STAR, radius=4, steps=0)
    assert np.array_equal(zero, x)


def test_translation_equivariance_periodic():
    """S_k(roll(x, t)) = roll(S_{roll(k, -t)}(x), t), bit-exact."""
    g = rng(16)
    x = g.uniform(-1, 1, (5, 6, 7))
    w = g.uniform(-1, 1, 27)
    k = g.uniform(0.5, 1, x.shape)
    t = (2, -1, 3)
    ax = (0, 1, 2)
    lhs = oracle.apply(np.roll(x, t, ax), w, shape=BOX, radius=1, boundary=PERIODIC, field=k)
    rhs = np.roll(oracle.apply(x, w, shape=BOX, radius=1, boundary=PERIODIC,
                               field=np.roll(k, tuple(-v for v in t), ax)), t, ax)
    assert np.array_equal(lhs, rhs)


def test_reflection():
    """S_w(flip x) = flip S_{flip w}(x): flipping the grid flips the kernel."""
    g = rng(17)
    x = g.uniform(-1, 1, (5, 6, 7))
    w = g.uniform(-1, 1, 27)
    wf = box_kernel(w, 3, 1)[::-1, ::-1, ::-1].ravel()
    for boundary in (ZERO, PERIODIC):
        lhs = oracle.apply(x[::-1, ::-1, ::-1], w, shape=BOX, radius=1, boundary=boundary, steps=2)
        rhs = oracle.apply(x, wf, shape=BOX, radius=1, boundary=boundary, steps=2)[::-1, ::-1, ::-1]
        np.testing.assert_allclose(lhs, rhs, rtol=0, atol=1e-13)


def test_zero_and_periodic_agree_inside():
    g = rng(18)
    x = g.uniform(-1, 1, (20, 21, 22))
    w = g.uniform(-1, 1, 13)
    R, s = 2, 3
    a = oracle.apply(x, w, shape=STAR, radius=R, boundary=ZERO, steps=s)
    b = oracle.apply(x, w, shape=STAR, radius=R, boundary=PERIODIC, steps=s)
    h = R * s
    inner = (slice(h, -h),) * 3
    assert np.array_equal(a[inner], b[inner])
    assert not np.allclose(a, b)


def test_linearity_and_norm_bound():
    g = rng(19)
    x1 = g.uniform(-1, 1, (6, 7, 8))
    x2 = g.uniform(-1, 1, (6, 7, 8))
    w = g.uniform(-1, 1, 27)
    w /= np.abs(w).sum()
    k = g.uniform(0.5, 1, x1.shape)
    f = lambda v: oracle.apply(v, w, shape=BOX, radius=1, boundary=PERIODIC, steps=2, field=k)
    np.testing.assert_allclose(f(2.0 * x1 - 3.0 * x2), 2.0 * f(x1) - 3.0 * f(x2), atol=1e-13)
    assert np.abs(f(x1)).max() <= np.abs(x1).max() + 1e-15


# ----------------------------------------------------------------------------- brute force

def dense_operator(dims, shape, R, w, boundary, k=None):
    """A[p, q] = sum over offsets o with bnd(p + o) = q of k[p] * w_o, built pair by pair."""
    off = oracle.offsets(shape, len(dims), R)
    dims3 = dims if len(dims) == 3 else (1,) + tuple(dims)
    n = int(np.prod(dims3))
    A = np.zeros((n, n))
    for p in itertools.product(*[range(d) for d in dims3]):
        ip = np.ravel_multi_index(p, dims3)
        for wj, o in zip(w, off):
            q = [p[a] + o[a] for a in range(3)]
            if boundary == ZERO:
                if any(q[a] < 0 or q[a] >= dims3[a] for a in range(3)):
                    continue
            else:
                q = [q[a] % dims3[a] for a in range(3)]
            A[ip, np.ravel_multi_index(q, dims3)] += wj * (1.0 if k is None else k.ravel()[ip])
    return A


@pytest.mark.parametrize("dims,shape,R", [((3, 4, 5), BOX, 1), ((5, 6), BOX, 2),
                                          ((4, 3, 6), STAR, 2), ((9, 9), STAR, 1)])
@pytest.mark.parametrize("boundary", [ZERO, PERIODIC])
def test_dense_matrix_power(dims, shape, R, boundary):
    g = rng(20)
    ndim = len(dims)
    x = g.uniform(-1, 1, dims)
    w = g.uniform(-1, 1, oracle.num_points(shape, ndim, R))
    k = g.uniform(0.5, 1, dims)
    A = dense_operator(dims, shape, R, w, boundary, k)
    steps = 3
    ref = np.linalg.matrix_power(A, steps) @ x.ravel()
    got = oracle.apply(x, w, shape=shape, radius=R, boundary=boundary, steps=steps, field=k,
                       ndim=ndim)
    np.testing.assert_allclose(got.ravel(), ref, rtol=0, atol=1e-13)


# ----------------------------------------------------------------------------- point sampler

@pytest.mark.parametrize("ndim,dims,shape,R,steps", [
    (3, (7, 8, 9), STAR, 4, 2), (3, (5, 6, 7), BOX, 1, 3), (2, (11, 13), BOX, 3, 2),
    (2, (6, 5), STAR, 1, 4), (3, (3, 2, 4), BOX, 2, 2)])
@pytest.mark.parametrize("boundary", [ZERO, PERIODIC])
def test_points_match_full(ndim, dims, shape, R, steps, boundary):
    g = rng(21)
    C, N = 2, 2
    x = g.uniform(-1, 1, (N * C,) + dims)
    k = g.uniform(0.5, 1, x.shape)
    w = g.uniform(-1, 1, (C, oracle.num_points(shape, ndim, R)))
    full = oracle.apply(x, w, shape=shape, radius=R, boundary=boundary, steps=steps, field=k,
                        ndim=ndim, channels=C)
    idx = np.array(list(itertools.product(range(N * C), *[range(d) for d in dims])))
    if ndim == 2:
        idx = np.concatenate([idx[:, :1], np.zeros((len(idx), 1), np.int64), idx[:, 1:]], 1)
    vals = oracle.apply_points(x, w, idx, shape=shape, radius=R, boundary=boundary, steps=steps,
                               field=k, ndim=ndim, channels=C)
    np.testing.assert_allclose(vals, full.ravel(), rtol=0, atol=1e-13)


def test_rejects_bad_arguments():
    x = np.zeros((3, 3, 3))
    with pytest.raises(ValueError):
        oracle.apply(x, np.zeros(27), shape=BOX, radius=1, steps=-1)
    with pytest.raises(ValueError):
        oracle.apply(x, np.zeros(27), shape=BOX, radius=1, boundary=5)
    with pytest.raises(ValueError):
        oracle.apply(x, np.zeros(26), shape=BOX, radius=1)
    with pytest.raises(ValueError):
        oracle.apply_points(x, np.zeros(27), [[0, 3, 0, 0]], shape=BOX, radius=1)


@pytest.mark.parametrize("shape", [STAR, BOX])
@pytest.mark.parametrize("boundary", [ZERO, PERIODIC])
def test_radius_zero_is_pointwise_scaling(shape, boundary):
    """Radius 0 (the degenerate stencil: one offset, the centre) reduces every step to
    u <- k * w0 * u, so s steps give (k w0)^s * u, with no neighbour and no boundary
    effect; per channel for batched volumes."""
    g = np.random.default_rng(31)
    C = 3
    x = g.uniform(-1, 1, (2 * C, 4, 5, 6))
    w = g.uniform(-1, 1, (C, 1))
    k = g.uniform(0.5, 1.0, x.shape)
    got = oracle.apply(x, w, shape=shape, radius=0, boundary=boundary, steps=3, field=k,
                       ndim=3, channels=C)
    scale = np.repeat(w[:, 0], 1)[np.arange(2 * C) % C][:, None, None, None]
    ref = (k * scale) ** 3 * x
    assert np.allclose(got, ref, rtol=1e-14, atol=1e-15)
