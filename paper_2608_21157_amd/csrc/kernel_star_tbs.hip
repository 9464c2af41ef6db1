// kernel_star_tbs.hip -- S star steps fused in one pass (temporal blocking), 3D, for
// radii with (S - 1) R <= the elements of one 16-byte vector; built for radius 1 with
// S = 3 and 4 (fp32) and S = 3 (fp64), gfx950.
//
// Computes u_S = S(...S(u_0)) for the star operator (centre plus -R..-1, +1..+R along z, y
// and x; cross-correlation as in the HIERA "Case-study protocol", generalised to stars,
// periodic wrap and batched volumes), reading u_0 and writing u_S once.  Under the zero
// boundary every intermediate u_k is zero outside the grid, as if written and re-read.
//
// A workgroup owns a TXV-vector x TYW-row tile of the x-y plane and streams a chunk of z
// planes.  Every thread owns one column of the stage-1 region: the tile plus B = (S-1) R
// rows above and below and one vector left and right.  Every thread evaluates every stage
// on its column; stage k lags stage k - 1 by R planes.  What a stage computes is exact on
// a region that shrinks by R rows per stage and, inside the side vectors, by R elements
// per stage, so stage S is exact on the tile as long as (S - 1) R fits one vector; values
// outside a stage's exact region are never read by an exact value of the next stage.
// Per stage a z-queue of its input (2R + 1 planes, plus a prefetched plane for u_0) lives
// in registers, and the input's current plane is staged in LDS (one barrier per plane,
// double-buffered).  u_0 cells beyond the region that stage 1 reads (R rows above and
// below, one more vector left and right) are loaded one plane ahead into registers.
//
// Against two fused steps (kernel_star_tb.hip) this moves half the HBM bytes per step
// and evaluates about 22% more columns per step, with one workgroup per CU (its LDS
// planes) instead of two.  Measured on MI355X, fp32 radius 1, 10 steps: 512^3 (beyond
// the Infinity Cache) 1235 -> 1406-1471 Gpoints/s with four steps per pass; 256^3
// (resident in it) 1300 -> 1230, so the planner fuses four steps only for working sets
// larger than the Infinity Cache.  Five steps (12 waves, 168 VGPRs) spill to scratch.
// fp64 radius 1, three steps per pass, 512^3, 9 steps: 507 -> 770-784 Gpoints/s against
// two.  fp32 radius 2 with three steps measured 2% slower than two and is not built.
#include "common.hpp"
#include "plan.hpp"

namespace stencil {
namespace {

struct TbsParams {
    int nz, ny, nx;
    long long vol;
    int ntx, nty;
    int zc, nzc;
    int nblocks;
    int channels;
};

template <typename T, int R, int S>
struct TbsShape {
    static constexpr int VEC = Vec16<T>::N;
    static constexpr int TXV = 16;                  // tile width in vectors
    static constexpr int TYW = 32;                  // tile height in rows
    static constexpr int B = (S - 1) * R;           // band rows above and below the tile
    static constexpr int CW = TXV + 2;              // region width: one vector each side
    static constexpr int CH = TYW + 2 * B;          // region height
    static constexpr int NCOL = CW * CH;
    static constexpr int THREADS = ((NCOL + 63) / 64) * 64;
    // LDS rectangle of every plane: rows -B-R .. TYW-1+B+R, vectors -2 .. TXV+1
    static constexpr int W = TXV + 4, H = CH + 2 * R;
    static constexpr int CELLS = H * W;
    // u_0 cells stage 1 reads beyond the region: R rows above and below (region width),
    // and the vectors -2 and TXV+1 on the region's rows
    static constexpr int NX_TB = 2 * R * CW;
    static constexpr int NX_LR = 2 * CH;
    static constexpr int NEX = (NX_TB + NX_LR + THREADS - 1) / THREADS;
    static constexpr int PF = 1;
    static constexpr int NQ = 2 * R + 1 + PF;
    static_assert(S >= 2, "at least two fused steps");
    static_assert((S - 1) * R <= VEC, "the side vector must hold the shrinking halo");
    static_assert(NQ % 2 == 0, "buffer parity follows the phase");
};

template <typename T, int R, int S, bool PERIODIC, int STORE_CP>
__global__ __launch_bounds__((TbsShape<T, R, S>::THREADS)) void stencil_star_tbs_kernel(
    const T *__restrict__ in, T *__restrict__ out, const T *__restrict__ w, TbsParams p)
{
    using SH = TbsShape<T, R, S>;
    constexpr int VEC = SH::VEC, TXV = SH::TXV, TYW = SH::TYW, B = SH::B, NQ = SH::NQ;
    constexpr int W = SH::W, CELLS = SH::CELLS, PF = SH::PF;
    constexpr int E = sizeof(T);
    // two sets of S planes, each with 64 spare cells (lanes with no cell write there)
    __shared__ Vec16<T> lds[2][S][CELLS + 64];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    int t = xcd_logical_block(blockIdx.x, p.nblocks);
    const int tx = t % p.ntx;
    t /= p.ntx;
    const int ty = t % p.nty;
    t /= p.nty;
    const int zi = t % p.nzc;
    const long long b = t / p.nzc;
    const int x0 = tx * TXV * VEC, y0 = ty * TYW;
    const long long plane = (long long)p.ny * p.nx;
    const unsigned plane_bytes = unsigned(plane * E);
    const T *src = in + b * p.vol;
    T *dst = out + b * p.vol;

    // ---- this thread's column (tile-relative row r, vector v) -----------------------
    const bool col = tid < SH::NCOL;
    const int r = col ? tid / SH::CW - B : 0;
    const int v = col ? tid % SH::CW - 1 : 0;
    const int gy = y0 + r, gx = x0 + v * VEC;
    const bool inside = col && gy >= 0 && gy < p.ny && gx >= 0 && gx < p.nx;
    const bool tile = col && r >= 0 && r < TYW && v >= 0 && v < TXV;
    auto goff = [&](int yy, int xx) {
        if (PERIODIC)
            return (wrap_index(yy, p.ny) * p.nx + wrap_index(xx, p.nx)) * E;
        return (yy >= 0 && yy < p.ny && xx >= 0 && xx < p.nx) ? (yy * p.nx + xx) * E
                                                               : kOutOfRange;
    };
    auto cell = [&](int rr, int vv) { return (rr + B + R) * W + (vv + 2); };
    const int qoff = col ? goff(gy, gx) : kOutOfRange;
    const int soff = (tile && inside) ? (gy * p.nx + gx) * E : kOutOfRange;
    const int idx = cell(r, v);
    const int wcell = col ? idx : CELLS + lane;

    int xoff[SH::NEX], xidx[SH::NEX];
#pragma unroll
    for (int h = 0; h < SH::NEX; ++h) {
        int j = tid + h * SH::THREADS;
        int rr = 0, vv = 0;
        bool any = true;
        if (j < SH::NX_TB) {
            const int k = j / SH::CW;
            rr = k < R ? -B - R + k : TYW + B + k - R;
            vv = j % SH::CW - 1;
        } else if ((j -= SH::NX_TB) < SH::NX_LR) {
            rr = j / 2 - B;
            vv = (j % 2 == 0) ? -2 : TXV + 1;
        } else {
            any = false;
        }
        xidx[h] = any ? cell(rr, vv) : CELLS + lane;
        xoff[h] = any ? goff(y0 + rr, x0 + vv * VEC) : kOutOfRange;
    }

    // ---- weights: z by queue position (direction-aware), y and x by offset -------------
    const T *wb = w + (b % p.channels) * (1 + 6 * R);
    const int dir = (zi & 1) ? -1 : 1;
    T wz[2 * R + 1], wy[2 * R], wx[2 * R];
    wz[R] = wb[0];
#pragma unroll
    for (int i = 0; i < 2 * R; ++i) {
        const int oz = i < R ? i - R : i - R + 1;
        const int pos = R + dir * oz;
#pragma unroll
        for (int q = 0; q < 2 * R + 1; ++q)
            if (q == pos)
                wz[q] = wb[1 + i];
        wy[i] = wb[1 + 2 * R + i];
        wx[i] = wb[1 + 4 * R + i];
    }

    // ---- z range: stage S writes [z0, z0 + n); stage 1 runs B planes ahead ------------
    const int z0 = zi * p.zc;
    const int n = min(p.zc, p.nz - z0);
    const int zs1 = dir > 0 ? z0 - B : z0 + n - 1 + B;  // stage-1 plane of iteration 0
    const int iters = n + 2 * B;

    auto plane_rsrc = [&](int z) {
        if (PERIODIC)
            return make_rsrc(src + wrap_index(z, p.nz) * plane, plane_bytes);
        // a plane outside the grid keeps its address (never dereferenced: zero records),
        // which leaves the address affine in the iteration, without a select
        const bool ok = unsigned(z) < unsigned(p.nz);  // 0 <= z < nz
        return make_rsrc(src + (long long)z * plane, ok ? plane_bytes : 0u);
    };
    auto z_inside = [&](int z) { return PERIODIC || unsigned(z) < unsigned(p.nz); };

    // ---- queues: position i of iteration m (phase m mod NQ) is slot (phase + i) mod NQ.
    // q[0] position i: u_0 at z1 + dir (i - R), i = 0 .. 2R + PF (the last PF prefetched);
    // q[k] position i: u_k at z_{k+1} + dir (i - R), i = 0 .. 2R, z_{k+1} = z1 - dir k R.
    Vec16<T> q[S][NQ], xr[2][SH::NEX];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const auto rx = plane_rsrc(zs1 + dir * k);
#pragma unroll
        for (int h = 0; h < SH::NEX; ++h)
            xr[k][h] = bload16<T>(rx, xoff[h]);
    }
#pragma unroll
    for (int i = 0; i < NQ; ++i) {
        q[0][i] = bload16<T>(plane_rsrc(zs1 + dir * (i - R)), qoff);
#pragma unroll
        for (int k = 1; k < S; ++k)
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                q[k][i].e[e] = T(0);
    }

    // one star evaluation of a column: z from its queue, y and x from the LDS plane
    auto stencil_at = [&](const Vec16<T> *buf, const Vec16<T>(&qq)[NQ], int phase)
        __attribute__((always_inline)) {
        Vec16<T> g[2 * R + 2];
#pragma unroll
        for (int i = 0; i < R; ++i) {
            g[i] = buf[idx + (i - R) * W];
            g[R + i] = buf[idx + (i + 1) * W];
        }
        g[2 * R] = buf[idx - 1];
        g[2 * R + 1] = buf[idx + 1];
        const Vec16<T> c = qq[(phase + R) % NQ];
        T acc[VEC];
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            acc[e] = wz[R] * c.e[e];
#pragma unroll
        for (int i = 0; i < 2 * R + 1; ++i) {
            if (i == R)
                continue;
            const Vec16<T> u = qq[(phase + i) % NQ];
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                acc[e] = fma(wz[i], u.e[e], acc[e]);
        }
#pragma unroll
        for (int i = 0; i < 2 * R; ++i)
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                acc[e] = fma(wy[i], g[i].e[e], acc[e]);
        T xs[3 * VEC];
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            xs[e] = g[2 * R].e[e];
            xs[VEC + e] = c.e[e];
            xs[2 * VEC + e] = g[2 * R + 1].e[e];
        }
#pragma unroll
        for (int i = 0; i < 2 * R; ++i) {
            const int ox = i < R ? i - R : i - R + 1;
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                acc[e] = fma(wx[i], xs[VEC + e + ox], acc[e]);
        }
        Vec16<T> res;
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            res.e[e] = acc[e];
        return res;
    };

    auto step = [&](int m, int phase) __attribute__((always_inline)) {
        const int buf = phase & 1;
        const int z1 = zs1 + dir * m;
        // stage the input plane of every stage and u_0's extra cells
#pragma unroll
        for (int k = 0; k < S; ++k)
            lds[buf][k][wcell] = q[k][(phase + R) % NQ];
#pragma unroll
        for (int h = 0; h < SH::NEX; ++h)
            lds[buf][0][xidx[h]] = xr[buf][h];
        {
            const auto rx = plane_rsrc(z1 + 2 * dir);
#pragma unroll
            for (int h = 0; h < SH::NEX; ++h)
                xr[buf][h] = bload16<T>(rx, xoff[h]);
        }
        __syncthreads();
        // stages 1 .. S; stage k computes u_k at z_k = z1 - dir (k - 1) R
#pragma unroll
        for (int k = 1; k <= S; ++k) {
            Vec16<T> u = stencil_at(lds[buf][k - 1], q[k - 1], phase);
            const int zk = z1 - dir * (k - 1) * R;
            if (!PERIODIC) {
                const bool keep = inside && z_inside(zk);
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    u.e[e] = keep ? u.e[e] : T(0);
            }
            if (k < S) {
                q[k][(phase + 2 * R) % NQ] = u;
            } else {
                // before the last stage has a full queue every lane's offset is out of
                // range, so plane zk's address (then possibly outside the grid) is unused
                const bool full = m >= 2 * B;
                bstore16<T, STORE_CP>(make_rsrc(dst + (long long)zk * plane, plane_bytes),
                                      full ? soff : kOutOfRange, u);
            }
        }
        q[0][phase] = bload16<T>(plane_rsrc(z1 + dir * (R + PF + 1)), qoff);
    };

    int m0 = 0;
    for (; m0 + NQ <= iters; m0 += NQ) {
#pragma unroll
        for (int ph = 0; ph < NQ; ++ph)
            step(m0 + ph, ph);
    }
#pragma unroll
    for (int ph = 0; ph < NQ - 1; ++ph)
        if (m0 + ph < iters)
            step(m0 + ph, ph);
}

template <typename T, int R, int S>
TbsParams make_params(const Geometry &g, int resident)
{
    using SH = TbsShape<T, R, S>;
    TbsParams p{};
    p.nz = int(g.nz);
    p.ny = int(g.ny);
    p.nx = int(g.nx);
    p.vol = g.vol;
    p.ntx = int((g.nx + SH::TXV * SH::VEC - 1) / (SH::TXV * SH::VEC));
    p.nty = int((g.ny + SH::TYW - 1) / SH::TYW);
    p.channels = g.channels;
    const long long base = g.batch * p.ntx * p.nty;
    const long long target = scaled_target(resident, g.grid_scale);
    long long nzc = (target + base - 1) / base;
    const long long min_len = 4 * SH::B;
    const long long max_chunks = (p.nz + min_len - 1) / min_len;
    if (nzc > max_chunks)
        nzc = max_chunks;
    if (nzc < 1)
        nzc = 1;
    p.zc = int((p.nz + nzc - 1) / nzc);
    p.nzc = (p.nz + p.zc - 1) / p.zc;
    p.nblocks = int(base * p.nzc);
    return p;
}

template <typename T, int R, int S, bool PERIODIC, int CP>
hipError_t launch_bc(const Geometry &g, const void *src, void *dst, const void *w,
                     hipStream_t stream)
{
    using SH = TbsShape<T, R, S>;
    const auto kernel = stencil_star_tbs_kernel<T, R, S, PERIODIC, CP>;
    static const int resident = resident_blocks(kernel, SH::THREADS);
    const TbsParams p = make_params<T, R, S>(g, resident);
    kernel<<<dim3(p.nblocks), dim3(SH::THREADS), 0, stream>>>(
        static_cast<const T *>(src), static_cast<T *>(dst), static_cast<const T *>(w), p);
    return hipGetLastError();
}

template <typename T, int R, int S>
hipError_t launch_s(const Geometry &g, const void *src, void *dst, const void *w,
                    hipStream_t stream)
{
    const bool per = g.boundary == STENCIL_PERIODIC;
    if (streaming_stores(g))
        return per ? launch_bc<T, R, S, true, kNonTemporal>(g, src, dst, w, stream)
                   : launch_bc<T, R, S, false, kNonTemporal>(g, src, dst, w, stream);
    return per ? launch_bc<T, R, S, true, 0>(g, src, dst, w, stream)
               : launch_bc<T, R, S, false, 0>(g, src, dst, w, stream);
}

}  // namespace

bool star_tbs_supported(const Geometry &g)
{
    return g.ndim == 3 && g.radius == 1 && star_stream_supported(g);
}

int star_tbs_max_depth(const Geometry &g)
{
    // (S - 1) R within one 16-byte vector: four floats, two doubles
    return g.dtype == STENCIL_F32 ? 4 : 3;
}

hipError_t launch_star_tbs(const Geometry &g, const void *src, void *dst, const void *w,
                           int depth, hipStream_t stream)
{
    if (!star_tbs_supported(g))
        return hipErrorInvalidValue;
    if (g.dtype == STENCIL_F64)
        return depth == 3 ? launch_s<double, 1, 3>(g, src, dst, w, stream) : hipErrorInvalidValue;
    switch (depth) {
    case 3: return launch_s<float, 1, 3>(g, src, dst, w, stream);
    case 4: return launch_s<float, 1, 4>(g, src, dst, w, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace stencil
