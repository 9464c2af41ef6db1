/*
 * oracle.c -- plain fp64 reference of the structured-grid stencil operator.
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the cpu_baseline
 * leg of bench.py load this file's library.  The HIP library never links, loads or calls
 * it, and it shares no code, header, table or constant with the HIP library.
 *
 * What it computes (HIERA, Sec. "Implementation and Evaluation Protocol", paragraph
 * "Case-study protocol"): a box stencil of radius R is a zero-padded cross-correlation
 * with padding R and stride 1, applied repeatedly to its own output, in FP64.  The
 * operator is generalised along the axes the five evaluated workloads need:
 *   - 2D or 3D grids, row-major, the last axis unit-stride;
 *   - STAR (centre + 2R points per axis) or BOX ((2R+1)^ndim points) offset sets;
 *   - ZERO boundary (every read outside the grid returns 0, at every step) or
 *     PERIODIC boundary (indices taken modulo the extent, non-negative modulo);
 *   - an optional coefficient field k indexed by the OUTPUT point:
 *       out[p] = sum_o k[p] * w[o] * in[p + o];
 *   - a batch of independent volumes, volume b using weight set (b mod channels).
 * One step is  u_{t+1}[p] = (k[p] *) sum_j w[j] * u_t(p + O[j]),  summed in offset
 * order j = 0, 1, ...  The result of `steps` steps is returned; steps = 0 copies.
 *
 * Offset order (the order of the weight vector):
 *   BOX : lexicographic over (oz, oy, ox), each from -R to +R, ox fastest
 *         (2D: (oy, ox)); weight j equals a correlation kernel entry [oz+R][oy+R][ox+R].
 *   STAR: the centre first; then for each axis from slowest to fastest the offsets
 *         -R..-1 followed by +1..+R along that axis.
 *
 * Plain loop nest, one thread, no blocking, fusion or reordering.  Build with
 * -O2 -fno-fast-math so that the sum order above is the one executed.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORACLE_STAR = 0, ORACLE_BOX = 1 };
enum { ORACLE_ZERO = 0, ORACLE_PERIODIC = 1 };

/* Number of stencil points: STAR 1 + 2*ndim*R, BOX (2R+1)^ndim.  -1 on bad input. */
int oracle_num_points(int shape, int ndim, int radius)
{
    if ((ndim != 2 && ndim != 3) || radius < 0)
        return -1;
    if (shape == ORACLE_STAR)
        return 1 + 2 * ndim * radius;
    if (shape == ORACLE_BOX) {
        int side = 2 * radius + 1, n = 1;
        for (int a = 0; a < ndim; ++a)
            n *= side;
        return n;
    }
    return -1;
}

/* Write the offsets in weight order as off[j][0..2] = (oz, oy, ox); oz = 0 in 2D. */
int oracle_offsets(int shape, int ndim, int radius, int32_t *off)
{
    int n = oracle_num_points(shape, ndim, radius);
    if (n < 0 || off == NULL)
        return -1;
    int j = 0;
    if (shape == ORACLE_BOX) {
        int zlo = (ndim == 3) ? -radius : 0, zhi = (ndim == 3) ? radius : 0;
        for (int oz = zlo; oz <= zhi; ++oz)
            for (int oy = -radius; oy <= radius; ++oy)
                for (int ox = -radius; ox <= radius; ++ox) {
                    off[3 * j + 0] = oz;
                    off[3 * j + 1] = oy;
                    off[3 * j + 2] = ox;
                    ++j;
                }
    } else {
        off[0] = off[1] = off[2] = 0;
        j = 1;
        /* axis index in (z, y, x); a 2D grid uses only y and x */
        for (int axis = (ndim == 3) ? 0 : 1; axis < 3; ++axis) {
            for (int r = -radius; r <= radius; ++r) {
                if (r == 0)
                    continue;
                off[3 * j + 0] = (axis == 0) ? r : 0;
                off[3 * j + 1] = (axis == 1) ? r : 0;
                off[3 * j + 2] = (axis == 2) ? r : 0;
                ++j;
            }
        }
    }
    return (j == n) ? 0 : -1;
}

static int64_t pmod(int64_t a, int64_t n)
{
    int64_t m = a % n;
    return (m < 0) ? m + n : m;
}

/* u(q) under the boundary rule; n[] are the (z, y, x) extents (nz = 1 in 2D). */
static double read_bnd(const double *u, const int64_t n[3], int boundary,
                       int64_t z, int64_t y, int64_t x)
{
    if (boundary == ORACLE_ZERO) {
        if (z < 0 || z >= n[0] || y < 0 || y >= n[1] || x < 0 || x >= n[2])
            return 0.0;
    } else {
        z = pmod(z, n[0]);
        y = pmod(y, n[1]);
        x = pmod(x, n[2]);
    }
    return u[(z * n[1] + y) * n[2] + x];
}

static int check_args(int ndim, const int64_t *dims, int64_t batch, int channels,
                      int shape, int radius, int boundary, int steps, int64_t n[3])
{
    if (ndim != 2 && ndim != 3)
        return -1;
    if (dims == NULL || batch < 1 || channels < 1 || steps < 0 || radius < 0)
        return -1;
    if (shape != ORACLE_STAR && shape != ORACLE_BOX)
        return -1;
    if (boundary != ORACLE_ZERO && boundary != ORACLE_PERIODIC)
        return -1;
    n[0] = (ndim == 3) ? dims[0] : 1;
    n[1] = (ndim == 3) ? dims[1] : dims[0];
    n[2] = (ndim == 3) ? dims[2] : dims[1];
    if (n[0] < 1 || n[1] < 1 || n[2] < 1)
        return -1;
    return 0;
}

/*
 * Full operator.  in/out: batch volumes, each dims-shaped, contiguous (volume b at
 * offset b * volume).  dims: (nz, ny, nx) in 3D, (ny, nx) in 2D.  w: channels * npts
 * weights in the order above.  field: NULL, or one dims-shaped coefficient field per
 * volume (same layout as in).  Returns 0, or -1 on bad arguments / allocation failure.
 */
int oracle_apply(const double *in, double *out, int ndim, const int64_t *dims,
                 int64_t batch, int channels, int shape, int radius, int boundary,
                 const double *w, const double *field, int steps)
{
    int64_t n[3];
    if (check_args(ndim, dims, batch, channels, shape, radius, boundary, steps, n) != 0)
        return -1;
    if (in == NULL || out == NULL || w == NULL)
        return -1;
    const int npts = oracle_num_points(shape, ndim, radius);
    int32_t *off = (int32_t *)malloc(sizeof(int32_t) * 3 * (size_t)npts);
    if (off == NULL)
        return -1;
    oracle_offsets(shape, ndim, radius, off);
    const int64_t vol = n[0] * n[1] * n[2];
    double *cur = (double *)malloc(sizeof(double) * (size_t)vol);
    double *nxt = (double *)malloc(sizeof(double) * (size_t)vol);
    if (cur == NULL || nxt == NULL) {
        free(off);
        free(cur);
        free(nxt);
        return -1;
    }

    for (int64_t b = 0; b < batch; ++b) {
        const double *wb = w + (size_t)(b % channels) * (size_t)npts;
        const double *kb = field ? field + b * vol : NULL;
        memcpy(cur, in + b * vol, sizeof(double) * (size_t)vol);
        for (int s = 0; s < steps; ++s) {
            for (int64_t z = 0; z < n[0]; ++z)
                for (int64_t y = 0; y < n[1]; ++y)
                    for (int64_t x = 0; x < n[2]; ++x) {
                        const int64_t p = (z * n[1] + y) * n[2] + x;
                        double acc = 0.0;
                        for (int j = 0; j < npts; ++j) {
                            const double v = read_bnd(cur, n, boundary, z + off[3 * j],
                                                      y + off[3 * j + 1], x + off[3 * j + 2]);
                            if (kb)
                                acc += kb[p] * wb[j] * v;
                            else
                                acc += wb[j] * v;
                        }
                        nxt[p] = acc;
                    }
            double *t = cur;
            cur = nxt;
            nxt = t;
        }
        memcpy(out + b * vol, cur, sizeof(double) * (size_t)vol);
    }
    free(off);
    free(cur);
    free(nxt);
    return 0;
}

/*
 * The same operator evaluated at selected output points only, for grids too large for
 * the full loop nest.  pts: nsamples rows of (b, z, y, x) (z = 0 in 2D).  For each point
 * the dependence cone is evaluated on a local window: level 0 holds the input under the
 * boundary rule on the box of half-width R*steps around the point, and level t holds
 * step t on the box shrunk by R per axis.  Under ZERO, window points outside the grid
 * hold 0 at every level (the padding is re-applied at every step).  Under PERIODIC the
 * window holds the periodic extension: the field is read at the wrapped index and the
 * extension of a step equals the step of the extension, so no wrap is needed between
 * levels.  Returns 0 or -1.
 */
int oracle_apply_points(const double *in, int ndim, const int64_t *dims, int64_t batch,
                        int channels, int shape, int radius, int boundary,
                        const double *w, const double *field, int steps,
                        int64_t nsamples, const int64_t *pts, double *vals)
{
    int64_t n[3];
    if (check_args(ndim, dims, batch, channels, shape, radius, boundary, steps, n) != 0)
        return -1;
    if (in == NULL || w == NULL || (nsamples > 0 && (pts == NULL || vals == NULL)))
        return -1;
    const int npts = oracle_num_points(shape, ndim, radius);
    int32_t *off = (int32_t *)malloc(sizeof(int32_t) * 3 * (size_t)npts);
    if (off == NULL)
        return -1;
    oracle_offsets(shape, ndim, radius, off);
    const int64_t vol = n[0] * n[1] * n[2];
    /* per-axis radius: no z extent of the cone in 2D */
    const int64_t rad[3] = {(ndim == 3) ? radius : 0, radius, radius};
    int64_t side0[3];
    for (int a = 0; a < 3; ++a)
        side0[a] = 2 * rad[a] * steps + 1;
    const size_t wsize = (size_t)(side0[0] * side0[1] * side0[2]);
    double *lev = (double *)malloc(sizeof(double) * wsize);
    double *nxt = (double *)malloc(sizeof(double) * wsize);
    if (lev == NULL || nxt == NULL) {
        free(off);
        free(lev);
        free(nxt);
        return -1;
    }

    for (int64_t i = 0; i < nsamples; ++i) {
        const int64_t b = pts[4 * i], pz = pts[4 * i + 1], py = pts[4 * i + 2],
                      px = pts[4 * i + 3];
        if (b < 0 || b >= batch || pz < 0 || pz >= n[0] || py < 0 || py >= n[1] || px < 0 ||
            px >= n[2]) {
            free(off);
            free(lev);
            free(nxt);
            return -1;
        }
        const double *ub = in + b * vol;
        const double *wb = w + (size_t)(b % channels) * (size_t)npts;
        const double *kb = field ? field + b * vol : NULL;

        /* level 0: window [p - R*steps, p + R*steps] per axis */
        int64_t h[3], s[3];
        for (int a = 0; a < 3; ++a) {
            h[a] = rad[a] * steps;
            s[a] = 2 * h[a] + 1;
        }
        for (int64_t a = 0; a < s[0]; ++a)
            for (int64_t c = 0; c < s[1]; ++c)
                for (int64_t d = 0; d < s[2]; ++d)
                    lev[(a * s[1] + c) * s[2] + d] =
                        read_bnd(ub, n, boundary, pz - h[0] + a, py - h[1] + c, px - h[2] + d);

        for (int t = 1; t <= steps; ++t) {
            int64_t hn[3], sn[3];
            for (int a = 0; a < 3; ++a) {
                hn[a] = rad[a] * (steps - t);
                sn[a] = 2 * hn[a] + 1;
            }
            for (int64_t a = 0; a < sn[0]; ++a)
                for (int64_t c = 0; c < sn[1]; ++c)
                    for (int64_t d = 0; d < sn[2]; ++d) {
                        /* global coordinates of this window point */
                        const int64_t gz = pz - hn[0] + a, gy = py - hn[1] + c,
                                      gx = px - hn[2] + d;
                        double acc = 0.0;
                        const int outside = gz < 0 || gz >= n[0] || gy < 0 || gy >= n[1] ||
                                            gx < 0 || gx >= n[2];
                        if (!(boundary == ORACLE_ZERO && outside)) {
                            double kp = 1.0;
                            if (kb)
                                kp = kb[(pmod(gz, n[0]) * n[1] + pmod(gy, n[1])) * n[2] +
                                        pmod(gx, n[2])];
                            for (int j = 0; j < npts; ++j) {
                                /* index of p + O[j] in the previous level's window */
                                const int64_t la = a + rad[0] + off[3 * j];
                                const int64_t lc = c + rad[1] + off[3 * j + 1];
                                const int64_t ld = d + rad[2] + off[3 * j + 2];
                                const double v = lev[(la * s[1] + lc) * s[2] + ld];
                                if (kb)
                                    acc += kp * wb[j] * v;
                                else
                                    acc += wb[j] * v;
                            }
                        }
                        nxt[(a * sn[1] + c) * sn[2] + d] = acc;
                    }
            double *tmp = lev;
            lev = nxt;
            nxt = tmp;
            for (int a = 0; a < 3; ++a) {
                h[a] = hn[a];
                s[a] = sn[a];
            }
        }
        vals[i] = lev[0];
    }
    free(off);
    free(lev);
    free(nxt);
    return 0;
}
