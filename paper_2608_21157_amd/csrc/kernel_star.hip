// kernel_star.hip -- star stencils of radius R <= 4 (1 + 6R points in 3D, 1 + 4R in 2D),
// 2.5D z-streaming with an LDS plane tile, gfx950.
//
// Computes one step of out[p] = sum_j w[j] * u(p + O[j]) over the star offsets (centre,
// then -R..-1, +1..+R along z, y and x) -- the operator of the HIERA case study ("Case-
// study protocol": zero-padded cross-correlation, stride 1), generalised to star offset
// sets, periodic wrap and batched volumes.
//
// Mapping:
//   * a workgroup (NW wavefronts) owns a TXW x TYW tile of the x-y plane and streams a
//     chunk of z planes; a lane owns a 16-byte vector along x times TY rows along y;
//   * z neighbours: every lane keeps the 2R + 1 planes around the current one for its own
//     points in registers (a queue of 2R + 1 + PF slots, PF of them prefetched planes),
//     so each input point is loaded from HBM once per chunk;
//   * x and y neighbours: the current plane is staged in LDS with an R-row halo above and
//     below and a whole-vector halo left and right (corners are never read by a star and
//     are not loaded); the halo is loaded one plane ahead into registers;
//   * LDS is double-buffered, one barrier per plane;
//   * consecutive z chunks of a column stream in opposite directions, so the R planes two
//     chunks share are read by both at about the same time (from L2, not twice from HBM);
//   * global accesses use buffer resources with 32-bit offsets; cells outside the grid
//     read zero (zero boundary) and stores outside the grid are dropped.
#include "common.hpp"
#include "plan.hpp"


namespace stencil {
namespace {


struct StarParams {
    int nz, ny, nx;
    long long vol;
    int ntx, nty;   // tiles along x and y
    int zc, nzc;    // planes per z chunk, chunks
    int nblocks;
    int channels;
};

template <typename T, int R, int TY, bool ZAXIS, int LX = 16, int NW = 4, int PF = 1>
struct StarShape {
    static constexpr int kLanesX = LX;                 // lanes along x in a row group
    static constexpr int kRowGroups = 64 / LX;         // row groups per wavefront
    static constexpr int kWaves = NW;                  // wavefronts per workgroup
    static constexpr int THREADS = 64 * NW;
    static constexpr int VEC = Vec16<T>::N;
    static constexpr int TXW = kLanesX * VEC;
    static constexpr int TYW = kWaves * kRowGroups * TY;
    static constexpr int HX = ((R + VEC - 1) / VEC) * VEC;  // x halo in whole vectors
    static constexpr int LDW = TXW + 2 * HX;                // LDS row pitch (elements)
    static constexpr int LDH = TYW + 2 * R;
    // queue slots: the 2R + 1 planes around the current one plus PF prefetched planes
    // (PF odd, so that the slot count is even and the LDS buffer parity stays static)
    static constexpr int NQ = ZAXIS ? 2 * R + 1 + PF : 1;
    static constexpr int NBUF = ZAXIS ? 2 : 1;
    // halo vectors per plane: R rows above and below (tile width), HX columns left/right
    static constexpr int HTB = 2 * R * (TXW / VEC);
    static constexpr int HLR = 2 * TYW * (HX / VEC);
    static constexpr int NH = (HTB + HLR + THREADS - 1) / THREADS;  // halo vectors per thread
};

template <typename T, int R, int TY, bool PERIODIC, bool ZAXIS, int STORE_CP, int LX, int NW,
          int PF>
__global__ __launch_bounds__(64 * NW) void stencil_star_stream_kernel(
    const T *__restrict__ in, T *__restrict__ out, const T *__restrict__ w, StarParams p)
{
    using S = StarShape<T, R, TY, ZAXIS, LX, NW, PF>;
    static_assert(!ZAXIS || S::NQ % 2 == 0, "queue length must be even");
    constexpr int kLanesX = S::kLanesX, kRowGroups = S::kRowGroups;
    constexpr int VEC = S::VEC, TXW = S::TXW, TYW = S::TYW, HX = S::HX, LDW = S::LDW;
    constexpr int NQ = S::NQ, NH = S::NH;
    constexpr int E = sizeof(T);
    constexpr int RZ = ZAXIS ? R : 0;
    // each LDS plane ends with 64 spare cells: a lane with no halo vector writes its
    // lane's spare cell, so the writes (and the loads feeding them) need no branch; a
    // load or store under a branch makes the compiler's wait counts conservative
    constexpr int SPARE = S::LDH * LDW / VEC;
    __shared__ Vec16<T> lds_raw[S::NBUF][SPARE + 64];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    int t = xcd_logical_block(blockIdx.x, p.nblocks);
    const int tx = t % p.ntx;
    t /= p.ntx;
    const int ty = t % p.nty;
    t /= p.nty;
    const int zi = t % p.nzc;
    const long long b = t / p.nzc;
    const int x0 = tx * TXW, y0 = ty * TYW;
    const int lxi = lane % kLanesX, rgi = lane / kLanesX;
    const int strip = (wave * kRowGroups + rgi) * TY;  // first own row within the tile
    const int x = x0 + lxi * VEC;
    const long long plane = (long long)p.ny * p.nx;
    const unsigned plane_bytes = unsigned(plane * E);
    const T *src = in + b * p.vol;
    T *dst = out + b * p.vol;

    // byte offset of the vector at grid row gy, column gx (a multiple of VEC): wrapped
    // under the periodic boundary, past the resource (reads zero) under the zero one
    auto goff = [&](int gy, int gx) {
        if (PERIODIC) {
            gy = wrap_index(gy, p.ny);
            gx = wrap_index(gx, p.nx);
            return (gy * p.nx + gx) * E;
        }
        return (gy >= 0 && gy < p.ny && gx >= 0 && gx < p.nx) ? (gy * p.nx + gx) * E
                                                               : kOutOfRange;
    };
    int own[TY], sto[TY];
#pragma unroll
    for (int o = 0; o < TY; ++o) {
        const int gy = y0 + strip + o;
        own[o] = goff(gy, x);
        sto[o] = (gy < p.ny && x < p.nx) ? (gy * p.nx + x) * E : kOutOfRange;
    }
    // halo vectors of this thread: global offset and LDS vector index (a spare cell: none)
    int hoff[NH], hlds[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) {
        const int idx = tid + S::THREADS * h;
        int ly = 0, lc = 0;
        hlds[h] = -1;
        hoff[h] = kOutOfRange;
        if (idx < S::HTB) {
            const int r = idx / (TXW / VEC);
            ly = r < R ? r : TYW + r;
            lc = HX + (idx % (TXW / VEC)) * VEC;
            hlds[h] = (ly * LDW + lc) / VEC;
        } else if (idx < S::HTB + S::HLR) {
            const int j = idx - S::HTB;
            const int per_row = 2 * (HX / VEC);
            const int k = j % per_row;
            ly = R + j / per_row;
            lc = (k < HX / VEC) ? k * VEC : TXW + k * VEC;  // left block, or right block
            hlds[h] = (ly * LDW + lc) / VEC;
        }
        if (hlds[h] >= 0)
            hoff[h] = goff(y0 + ly - R, x0 + lc - HX);
        else
            hlds[h] = SPARE + lane;
    }

    // weights: z by queue position (direction-aware), y and x by offset
    const T *wb = w + (b % p.channels) * (1 + 2 * (ZAXIS ? 3 : 2) * R);
    const int dir = (ZAXIS && (zi & 1)) ? -1 : 1;
    T wz[2 * RZ + 1], wy[2 * R], wx[2 * R];
    wz[RZ] = wb[0];
    int j = 1;
    if (ZAXIS) {
#pragma unroll
        for (int i = 0; i < 2 * R; ++i) {
            // weight index i is offset -R..-1, +1..+R; queue position of offset oz is
            // R + dir * oz
            const int oz = i < R ? i - R : i - R + 1;
            const int pos = R + dir * oz;
            // written with a select so that the array index stays static
#pragma unroll
            for (int q = 0; q < 2 * R + 1; ++q)
                if (q == pos)
                    wz[q] = wb[1 + i];
        }
        j += 2 * R;
    }
#pragma unroll
    for (int i = 0; i < 2 * R; ++i)
        wy[i] = wb[j + i];
#pragma unroll
    for (int i = 0; i < 2 * R; ++i)
        wx[i] = wb[j + 2 * R + i];

    const int z0 = zi * p.zc;
    const int n = min(p.zc, p.nz - z0);
    const int zs = dir > 0 ? z0 : z0 + n - 1;

    auto plane_rsrc = [&](int z) {
        if (PERIODIC)
            return make_rsrc(src + wrap_index(z, p.nz) * plane, plane_bytes);
        // a plane outside the grid keeps its address (never dereferenced: zero records),
        // which leaves the address affine in the iteration, without a select
        const bool ok = unsigned(z) < unsigned(p.nz);  // 0 <= z < nz
        return make_rsrc(src + (long long)z * plane, ok ? plane_bytes : 0u);
    };

    Vec16<T> Q[NQ][TY];
    Vec16<T> hreg[NH];
    // prologue: halo of zs, then queue positions 0 .. 2R + PF (planes zs + dir * (i - R)).
    // The halo goes first so that, at the loop head, as many loads follow it on the entry
    // path as in the steady state: the wait before its LDS write then stays partial.
    {
        const auto rh = plane_rsrc(zs);
#pragma unroll
        for (int h = 0; h < NH; ++h)
            hreg[h] = bload16<T>(rh, hoff[h]);
    }
#pragma unroll
    for (int i = 0; i < NQ; ++i) {
        const auto rq = plane_rsrc(zs + dir * (i - RZ));
#pragma unroll
        for (int o = 0; o < TY; ++o)
            Q[i][o] = bload16<T>(rq, own[o]);
    }

    // one plane: iteration m (phase = m mod NQ) computes output plane zs + dir * m
    auto step = [&](int m, int phase) {
        const int zc = zs + dir * m;
        Vec16<T> *buf = lds_raw[ZAXIS ? (phase & 1) : 0];
        // stage the current plane: own rows (queue position R) and the halo
#pragma unroll
        for (int o = 0; o < TY; ++o)
            buf[((R + strip + o) * LDW + HX + lxi * VEC) / VEC] = Q[(phase + RZ) % NQ][o];
#pragma unroll
        for (int h = 0; h < NH; ++h)
            buf[hlds[h]] = hreg[h];
        if (ZAXIS) {
            const auto rh = plane_rsrc(zc + dir);
#pragma unroll
            for (int h = 0; h < NH; ++h)
                hreg[h] = bload16<T>(rh, m + 1 < n ? hoff[h] : kOutOfRange);
        }
        __syncthreads();

        const auto rd = make_rsrc(dst + (long long)zc * plane, plane_bytes);
#pragma unroll
        for (int o = 0; o < TY; ++o) {
            const Vec16<T> c = Q[(phase + RZ) % NQ][o];
            T acc[VEC];
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                acc[e] = wz[RZ] * c.e[e];
            // z neighbours from the queue
#pragma unroll
            for (int i = 0; i < 2 * RZ + 1; ++i) {
                if (i == RZ)
                    continue;
                const Vec16<T> v = Q[(phase + i) % NQ][o];
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    acc[e] = fma(wz[i], v.e[e], acc[e]);
            }
            // y neighbours: own rows from the queue, the others from LDS
#pragma unroll
            for (int i = 0; i < 2 * R; ++i) {
                const int oy = i < R ? i - R : i - R + 1;
                const int row = o + oy;
                Vec16<T> v;
                if (row >= 0 && row < TY)
                    v = Q[(phase + RZ) % NQ][row];
                else
                    v = buf[((R + strip + row) * LDW + HX + lxi * VEC) / VEC];
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    acc[e] = fma(wy[i], v.e[e], acc[e]);
            }
            // x neighbours from the LDS row: HX elements each side
            T xs[2 * HX + VEC];
            const int rowbase = ((R + strip + o) * LDW + lxi * VEC) / VEC;
#pragma unroll
            for (int k = 0; k < HX / VEC; ++k) {
                const Vec16<T> l = buf[rowbase + k];
                const Vec16<T> r = buf[rowbase + (HX + VEC) / VEC + k];
#pragma unroll
                for (int e = 0; e < VEC; ++e) {
                    xs[k * VEC + e] = l.e[e];
                    xs[HX + VEC + k * VEC + e] = r.e[e];
                }
            }
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                xs[HX + e] = c.e[e];
#pragma unroll
            for (int i = 0; i < 2 * R; ++i) {
                const int ox = i < R ? i - R : i - R + 1;
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    acc[e] = fma(wx[i], xs[HX + e + ox], acc[e]);
            }
            Vec16<T> res;
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                res.e[e] = acc[e];
            bstore16<T, STORE_CP>(rd, sto[o], res);
        }
        // the slot of queue position 0 is free: prefetch plane zc + dir * (R + PF + 1),
        // which is first used PF + 1 planes from now
        if (ZAXIS) {
            const auto rq = plane_rsrc(zc + dir * (R + PF + 1));
#pragma unroll
            for (int o = 0; o < TY; ++o)
                Q[phase][o] = bload16<T>(rq, m + PF + 1 <= n - 1 ? own[o] : kOutOfRange);
        }
    };

    if (!ZAXIS) {
        step(0, 0);
        return;
    }
    // whole groups of NQ planes in the loop, the remainder after it: an early exit inside
    // the loop body would merge into the loop head and make its waits conservative
    int m0 = 0;
    for (; m0 + NQ <= n; m0 += NQ) {
#pragma unroll
        for (int ph = 0; ph < NQ; ++ph)
            step(m0 + ph, ph);
    }
#pragma unroll
    for (int ph = 0; ph < NQ - 1; ++ph)
        if (m0 + ph < n)
            step(m0 + ph, ph);
}

template <typename T, int R, int TY, bool ZAXIS, int LX, int NW>
StarParams make_params(const Geometry &g)
{
    using S = StarShape<T, R, TY, ZAXIS, LX, NW>;
    StarParams p{};
    p.nz = int(g.nz);
    p.ny = int(g.ny);
    p.nx = int(g.nx);
    p.vol = g.vol;
    p.ntx = int((g.nx + S::TXW - 1) / S::TXW);
    p.nty = int((g.ny + S::TYW - 1) / S::TYW);
    p.channels = g.channels;
    const long long base = g.batch * p.ntx * p.nty;
    long long nzc = 1;
    if (ZAXIS) {
        // enough workgroups for 256 CUs (scaled by the plan's grid_scale), with chunks of
        // at least 4 queue depths
        const long long target = scaled_target(256, g.grid_scale);
        nzc = (target + base - 1) / base;
        const long long min_len = 4 * (2 * R + 1);
        const long long max_chunks = (p.nz + min_len - 1) / min_len;
        if (nzc > max_chunks)
            nzc = max_chunks;
        if (nzc < 1)
            nzc = 1;
    }
    p.zc = int((p.nz + nzc - 1) / nzc);
    p.nzc = (p.nz + p.zc - 1) / p.zc;
    p.nblocks = int(base * p.nzc);
    return p;
}

template <typename T, int R, int TY, bool ZAXIS, int CP, int LX, int NW, int PF>
hipError_t launch_shape(const Geometry &g, const void *src, void *dst, const void *w,
                        hipStream_t stream)
{
    const StarParams p = make_params<T, R, TY, ZAXIS, LX, NW>(g);
    const T *s = static_cast<const T *>(src);
    T *d = static_cast<T *>(dst);
    const T *wt = static_cast<const T *>(w);
    if (g.boundary == STENCIL_PERIODIC)
        stencil_star_stream_kernel<T, R, TY, true, ZAXIS, CP, LX, NW, PF>
            <<<dim3(p.nblocks), dim3(64 * NW), 0, stream>>>(s, d, wt, p);
    else
        stencil_star_stream_kernel<T, R, TY, false, ZAXIS, CP, LX, NW, PF>
            <<<dim3(p.nblocks), dim3(64 * NW), 0, stream>>>(s, d, wt, p);
    return hipGetLastError();
}

// Tile shape, measured on MI355X (512^3, radius 4): 64 x 64 tiles (8 wavefronts) with one
// prefetched plane were the fastest of the 16/32/64-lane-wide, 4/8-wavefront and 1/3/5-plane
// prefetch variants (all within a few percent); 2D grids use 64 x 32 tiles for more tiles.
// The plan's tile selects 64 x 32 (tile 1) or 64 x 64 (tile 2) explicitly.
template <typename T, int R, int TY, bool ZAXIS, int CP>
hipError_t launch_cp(const Geometry &g, const void *src, void *dst, const void *w,
                     hipStream_t stream)
{
    const bool large = stream_tile(g, 1) == 2;
    if (large)
        return launch_shape<T, R, TY, ZAXIS, CP, 16, 8, 1>(g, src, dst, w, stream);
    return launch_shape<T, R, TY, ZAXIS, CP, 16, 4, 1>(g, src, dst, w, stream);
}

template <typename T, int R, int TY, bool ZAXIS>
hipError_t launch_r(const Geometry &g, const void *src, void *dst, const void *w,
                    hipStream_t stream)
{
    if (streaming_stores(g))
        return launch_cp<T, R, TY, ZAXIS, kNonTemporal>(g, src, dst, w, stream);
    return launch_cp<T, R, TY, ZAXIS, 0>(g, src, dst, w, stream);
}

template <typename T, bool ZAXIS>
hipError_t launch_t(const Geometry &g, const void *src, void *dst, const void *w,
                    hipStream_t stream)
{
    switch (g.radius) {
    case 1: return launch_r<T, 1, 2, ZAXIS>(g, src, dst, w, stream);
    case 2: return launch_r<T, 2, 2, ZAXIS>(g, src, dst, w, stream);
    case 3: return launch_r<T, 3, 2, ZAXIS>(g, src, dst, w, stream);
    case 4: return launch_r<T, 4, 2, ZAXIS>(g, src, dst, w, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace

bool star_stream_supported(const Geometry &g)
{
    if (g.shape != STENCIL_STAR || g.radius < 1 || g.radius > 4 || g.field)
        return false;
    const int vec = (g.dtype == STENCIL_F32) ? 4 : 2;
    if (g.nx % vec != 0)
        return false;
    // byte offsets within a plane stay below the out-of-range marker; blocks fit int
    return g.ny * g.nx * int64_t(g.elt) < (int64_t(1) << 30) &&
           g.batch * g.ny * g.nx < (int64_t(1) << 31);
}

hipError_t launch_star_stream(const Geometry &g, const void *src, void *dst, const void *w,
                              hipStream_t stream)
{
    const bool z = g.ndim == 3;
    if (g.dtype == STENCIL_F32)
        return z ? launch_t<float, true>(g, src, dst, w, stream)
                 : launch_t<float, false>(g, src, dst, w, stream);
    return z ? launch_t<double, true>(g, src, dst, w, stream)
             : launch_t<double, false>(g, src, dst, w, stream);
}

}  // namespace stencil
