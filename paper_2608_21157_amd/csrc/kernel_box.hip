// kernel_box.hip -- 27-point (3x3x3 box, radius 1) stencil, 2.5D z-streaming, gfx950.
//
// Computes one step of out[p] = (k[p] *) sum_o w[o] * in[p + o] over the 27 offsets
// o in [-1, 1]^3 (cross-correlation, HIERA "Case-study protocol", generalised to 3D with
// an output-indexed coefficient field, zero or periodic boundary, and batched volumes
// with per-channel weights).
//
// Mapping (no LDS, no barriers):
//   * a wavefront owns a row segment of 64 lanes x 16 bytes (256 floats / 128 doubles)
//     along x -- or, for narrower rows, 64/lpr whole rows side by side -- times TY rows
//     per lane along y, and streams a chunk of z planes (even chunks upwards, odd chunks
//     downwards, so neighbouring chunks read their shared halo plane at about the same time);
//   * every input plane is read once per wavefront as TY + 2 coalesced 16-byte row loads
//     per lane (the two extra rows are the y halo, shared through L2 with the wave that
//     owns them);
//   * x neighbours come from the adjacent lanes through DPP wave shifts; only the first
//     and last lane of a segment load the one-element x halo;
//   * each input row is folded into three rotating accumulator planes (the outputs at
//     z_in - 1, z_in, z_in + 1), so the completed plane z_in - 1 is written as soon as
//     plane z_in has been read;
//   * each row register is reloaded with the next plane right after its last use, so
//     the loads of plane z_in + 1 are in flight while plane z_in is folded in;
//   * loads and stores use buffer resources: 32-bit offsets, and rows outside the grid
//     take an offset past the resource, which reads zero (the zero padding) and drops
//     stores.
// Workgroups are 4 wavefronts stacked along y; their order is renumbered per XCD.
#include "common.hpp"
#include "plan.hpp"

#include <algorithm>
#include <type_traits>


namespace stencil {
namespace {

struct BoxParams {
    int nz, ny, nx;
    long long vol;
    int lpr;        // lanes per row segment, 2..64
    int segw;       // x extent of a segment = lpr * elements per 16 bytes
    int segs;       // segments per row
    int rows_wave;  // output rows per wavefront = (64 / lpr) * TY
    int ywaves;     // wavefront row blocks per volume
    int ygroups;    // workgroup row blocks per volume (4 wavefronts each)
    int zc, nzc;    // z planes per chunk, chunks per volume
    int channels;
    int nblocks;
};

template <typename T>
__device__ __forceinline__ T madd(T a, T b, T c)
{
    return fma(a, b, c);
}

template <typename T, int TY, bool PERIODIC, bool FIELD, int STORE_CP, int INNER_CP, bool XHALO>
__global__ __launch_bounds__(256) void stencil_box3_stream_kernel(
    const T *__restrict__ in, T *__restrict__ out, const T *__restrict__ field,
    const T *__restrict__ w, BoxParams p)
{
    constexpr int VEC = Vec16<T>::N;
    constexpr int NR = TY + 2;  // input rows per lane and plane
    constexpr int E = sizeof(T);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;

    // logical tile order: x segment fastest, then row block, then z chunk, then volume,
    // so that the segments of one row block (which read each other's x halo) and the
    // neighbouring row blocks run on the same XCD at about the same time
    int t = xcd_logical_block(blockIdx.x, p.nblocks);
    const int seg = t % p.segs;
    t /= p.segs;
    const int yg = t % p.ygroups;
    t /= p.ygroups;
    const int zi = t % p.nzc;
    const long long b = t / p.nzc;
    const int yw = yg * 4 + wave;
    if (yw >= p.ywaves)
        return;  // whole wavefront leaves; the kernel has no barriers

    const int lx = lane % p.lpr;
    const int rg = lane / p.lpr;
    const int x = seg * p.segw + lx * VEC;
    const int y0 = yw * p.rows_wave + rg * TY;
    const int z0 = zi * p.zc;
    const int n = min(p.zc, p.nz - z0);  // output planes of this chunk
    const long long plane = (long long)p.ny * p.nx;
    const unsigned plane_bytes = unsigned(plane * E);
    const T *src = in + b * p.vol;
    T *dst = out + b * p.vol;
    const T *kf = FIELD ? field + b * p.vol : nullptr;
    const T *wb = w + (b % p.channels) * 27;
    // Odd chunks stream downwards, so that two neighbouring chunks reach the plane they
    // share as a halo at about the same time (the second read then hits L2).  Streaming
    // down mirrors the z offsets: weight plane a is then applied as plane 2 - a.
    const bool up = (zi & 1) == 0;
    auto zin = [&](int k) { return up ? z0 - 1 + k : z0 + n - k; };   // input plane k
    auto zout = [&](int q) { return up ? z0 + q : z0 + n - 1 - q; };  // output plane q
    T W[27];
#pragma unroll
    for (int j = 0; j < 27; ++j)
        W[j] = wb[up ? j : (2 - j / 9) * 9 + j % 9];

    // byte offsets of input rows y0 - 1 .. y0 + TY within a plane; rows outside the grid
    // (zero boundary) get an offset past the resource and read as zero.  Without XHALO
    // (a segment is a whole row under the zero boundary) the x halo is the zero padding:
    // no halo loads and no halo registers
    const bool first = lx == 0, last = lx == p.lpr - 1;
    int hx = first ? seg * p.segw - 1 : seg * p.segw + p.segw;
    bool hok = (first || last) && hx >= 0 && hx < p.nx;
    if (PERIODIC) {
        hx = wrap_index(hx, p.nx);
        hok = first || last;
    }
    constexpr int NH = XHALO ? NR : 1;
    int ro[NR], ho[NH];
#pragma unroll
    for (int i = 0; i < NR; ++i) {
        int yi = y0 - 1 + i;
        bool ok = yi >= 0 && yi < p.ny;
        if (PERIODIC) {
            yi = wrap_index(yi, p.ny);
            ok = true;
        }
        ro[i] = ok ? (yi * p.nx + x) * E : kOutOfRange;
        if (XHALO)
            ho[i] = (ok && hok) ? (yi * p.nx + hx) * E : kOutOfRange;
    }

    // resource of input plane z_in; under the zero boundary a plane outside the grid
    // gets zero records, so every load from it returns zero
    auto plane_rsrc = [&](int zin) {
        bool zok = zin >= 0 && zin < p.nz;
        if (PERIODIC) {
            zin = wrap_index(zin, p.nz);
            zok = true;
        }
        return make_rsrc(src + (zok ? zin : 0) * plane, zok ? plane_bytes : 0u);
    };

    T acc[3][TY][VEC];
#pragma unroll
    for (int s = 0; s < 3; ++s)
#pragma unroll
        for (int o = 0; o < TY; ++o)
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                acc[s][o][e] = T(0);

    Vec16<T> rows[NR];
    T halo[NH];
    Vec16<T> kv[TY];
    {
        const auto r0 = plane_rsrc(zin(0));
#pragma unroll
        for (int i = 0; i < NR; ++i) {
            rows[i] = bload16<T>(r0, ro[i]);
            if (XHALO)
                halo[i] = bload1(r0, ho[i], T(0));
        }
    }
    auto load_field = [&](int q) {
        if (FIELD) {
            const auto rk = make_rsrc(kf + (long long)zout(q) * plane, plane_bytes);
#pragma unroll
            for (int o = 0; o < TY; ++o)
                kv[o] = bload16<T, kNonTemporal>(rk, ((y0 + o) * p.nx + x) * E);
        }
    };

    // Fold input plane k (z_in = zin(k)) into the accumulators, reloading each row
    // register with the next plane right after its last use.  Offset (a, bb, c) in the
    // (mirrored when streaming down) weight order is (oz, oy, ox) = (a - 1, bb - 1, c - 1);
    // the input point feeds output plane q = k - a (slot q mod 3, z = zout(q)) and output
    // row o = i - bb.  Planes q < 0 are skipped
    // (prologue only).
    // CHECK: skip output planes q < 0 (the prologue); in the steady state every q = k - a
    // is accumulated, since planes q >= n never complete and are never written (no branch
    // there keeps the loop free of conditional work).  With a coefficient field the
    // branch is kept (measured: c5 +1.2%, c5b +2.3% without it; c4, with the field, -1.3%).
    auto fold = [&](int k, auto slot_of_a, auto check) {
        const bool more = k + 1 <= n + 1;
        const auto rn = plane_rsrc(zin(k + 1));
#pragma unroll
        for (int i = 0; i < NR; ++i) {
            T r[VEC + 2];
            if constexpr (XHALO) {
                const T left = from_left_lane(rows[i].e[VEC - 1], halo[i]);
                const T right = from_right_lane(rows[i].e[0], halo[i]);
                r[0] = first ? halo[i] : left;
                r[VEC + 1] = last ? halo[i] : right;
            } else {
                const T left = from_left_lane_or_zero(rows[i].e[VEC - 1]);
                const T right = from_right_lane_or_zero(rows[i].e[0]);
                r[0] = first ? T(0) : left;
                r[VEC + 1] = last ? T(0) : right;
            }
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                r[e + 1] = rows[i].e[e];
            // unconditional (an offset past the resource after the last plane): a load
            // under a branch would make the compiler's wait counts conservative.  Rows
            // 2 .. TY - 1 are read by this wavefront only (no other one has them in its
            // halo) and may be streamed past the caches (INNER_CP)
            rows[i] = (i >= 2 && i <= TY - 1) ? bload16<T, INNER_CP>(rn, more ? ro[i] : kOutOfRange)
                                              : bload16<T>(rn, more ? ro[i] : kOutOfRange);
            if (XHALO)
                halo[i] = bload1(rn, more ? ho[i] : kOutOfRange, T(0));
#pragma unroll
            for (int a = 0; a < 3; ++a) {
                if (FIELD ? (k - a < 0 || k - a >= n) : (decltype(check)::value && k - a < 0))
                    continue;  // uniform with a field; else compile-time (prologue only)
                const int s = slot_of_a(a);
#pragma unroll
                for (int bb = 0; bb < 3; ++bb) {
                    const int o = i - bb;
                    if (o < 0 || o >= TY)
                        continue;  // resolved at compile time
                    const T w0 = W[a * 9 + bb * 3 + 0], w1 = W[a * 9 + bb * 3 + 1],
                            w2 = W[a * 9 + bb * 3 + 2];
#pragma unroll
                    for (int e = 0; e < VEC; ++e) {
                        T v = acc[s][o][e];
                        v = madd(w0, r[e], v);
                        v = madd(w1, r[e + 1], v);
                        v = madd(w2, r[e + 2], v);
                        acc[s][o][e] = v;
                    }
                }
            }
        }
    };

    // write output plane q from slot s (rows past the grid fall outside the resource and
    // are dropped) and clear the slot; the field rows are read here rather than prefetched,
    // which keeps the kernel at three wavefronts per SIMD
    auto emit = [&](int q, int s) {
        const auto rd = make_rsrc(dst + (long long)zout(q) * plane, plane_bytes);
        load_field(q);
#pragma unroll
        for (int o = 0; o < TY; ++o) {
            Vec16<T> v;
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                v.e[e] = FIELD ? acc[s][o][e] * kv[o].e[e] : acc[s][o][e];
            const int yo = y0 + o;
            bstore16<T, STORE_CP>(rd, yo < p.ny ? (yo * p.nx + x) * E : kOutOfRange, v);
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                acc[s][o][e] = T(0);
        }
    };

    // prologue: planes k = 0, 1 (no output plane completes yet)
    fold(0, [](int a) { return (3 - a) % 3; }, std::true_type{});
    fold(1, [](int a) { return (4 - a) % 3; }, std::true_type{});

    // steady state: plane k = 2 + 3m + j completes output plane q = k - 2 (slot j)
    for (int k0 = 2; k0 <= n + 1; k0 += 3) {
#pragma unroll
        for (int j = 0; j < 3; ++j) {
            const int k = k0 + j;
            if (k > n + 1)
                break;
            fold(k, [j](int a) { return (2 + j - a + 3) % 3; }, std::false_type{});
            emit(k - 2, j);
        }
    }
}

template <typename T>
constexpr int vec_of()
{
    return Vec16<T>::N;
}

int lanes_per_row(const Geometry &g, int vec)
{
    if (g.nx % vec != 0)
        return 0;
    const int64_t nxv = g.nx / vec;
    if (nxv >= 64)
        return (nxv % 64 == 0) ? 64 : 0;
    return (nxv >= 2 && 64 % nxv == 0) ? int(nxv) : 0;
}

template <typename T, int TY>
BoxParams make_params(const Geometry &g)
{
    constexpr int VEC = Vec16<T>::N;
    BoxParams p{};
    p.nz = int(g.nz);
    p.ny = int(g.ny);
    p.nx = int(g.nx);
    p.vol = g.vol;
    p.lpr = lanes_per_row(g, VEC);
    p.segw = p.lpr * VEC;
    p.segs = p.nx / p.segw;
    p.rows_wave = (64 / p.lpr) * TY;
    p.ywaves = (p.ny + p.rows_wave - 1) / p.rows_wave;
    p.ygroups = (p.ywaves + 3) / 4;
    p.channels = g.channels;
    const long long base = g.batch * p.segs * p.ygroups;
    // up to 16384 workgroups (64 per CU), in chunks of at least 8 planes; grid_scale
    // scales the workgroup target and, when positive, shortens the minimum chunk to
    // 8 >> grid_scale planes (at least 4).  Same-box A/B against 8192 workgroups of at
    // least 16 planes: 256 volumes of 128^3 fp32 0.7566 -> 0.7379 and 0.7605 -> 0.7403 ms
    // (8192 instead of 4096 workgroups), 64 volumes of 128^3 fp64 0.3601 -> 0.3573 ms,
    // 512^3 with a field level.
    const long long target = scaled_target(16384, g.grid_scale);
    long long nzc = (target + base - 1) / base;
    const long long min_len = g.grid_scale > 0 ? std::max(4, 8 >> g.grid_scale) : 8;
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

template <typename T, int TY, int CP, int ICP>
hipError_t launch_icp(const BoxParams &p, const Geometry &g, const void *src, void *dst,
                      const void *field, const void *w, hipStream_t stream)
{
    const T *s = static_cast<const T *>(src);
    T *d = static_cast<T *>(dst);
    const T *k = static_cast<const T *>(field);
    const T *wt = static_cast<const T *>(w);
    const dim3 grid(p.nblocks), block(256);
    const bool per = g.boundary == STENCIL_PERIODIC;
    // a whole row per segment under the zero boundary: the x halo is the padding
    const bool xhalo = per || p.segs > 1;
    if (per && g.field)
        stencil_box3_stream_kernel<T, TY, true, true, CP, ICP, true><<<grid, block, 0, stream>>>(s, d, k, wt, p);
    else if (per)
        stencil_box3_stream_kernel<T, TY, true, false, CP, ICP, true><<<grid, block, 0, stream>>>(s, d, k, wt, p);
    else if (g.field && xhalo)
        stencil_box3_stream_kernel<T, TY, false, true, CP, ICP, true><<<grid, block, 0, stream>>>(s, d, k, wt, p);
    else if (g.field)
        stencil_box3_stream_kernel<T, TY, false, true, CP, ICP, false><<<grid, block, 0, stream>>>(s, d, k, wt, p);
    else if (xhalo)
        stencil_box3_stream_kernel<T, TY, false, false, CP, ICP, true><<<grid, block, 0, stream>>>(s, d, k, wt, p);
    else
        stencil_box3_stream_kernel<T, TY, false, false, CP, ICP, false><<<grid, block, 0, stream>>>(s, d, k, wt, p);
    return hipGetLastError();
}

template <typename T, int TY, int CP>
hipError_t launch_cp(const Geometry &g, const void *src, void *dst, const void *field,
                     const void *w, hipStream_t stream)
{
    const BoxParams p = make_params<T, TY>(g);
    // Inner rows streamed past the caches when a wavefront owns full-width 64-lane row
    // segments and the output is streamed too (same-box A/B, Gpoints/s: 512^3 with a
    // field 495 -> 508, 128^3 fp64 volumes 341 -> 348); with several narrow rows per
    // wavefront it measured 2% slower (128^3 fp32 volumes: 698 -> 686)
    if constexpr (CP == kNonTemporal) {
        if (p.lpr == 64)
            return launch_icp<T, TY, CP, kNonTemporal>(p, g, src, dst, field, w, stream);
    }
    return launch_icp<T, TY, CP, 0>(p, g, src, dst, field, w, stream);
}

template <typename T, int TY>
hipError_t launch_ty(const Geometry &g, const void *src, void *dst, const void *field,
                     const void *w, hipStream_t stream)
{
    if (streaming_stores(g))
        return launch_cp<T, TY, kNonTemporal>(g, src, dst, field, w, stream);
    return launch_cp<T, TY, 0>(g, src, dst, field, w, stream);
}

}  // namespace

bool box_stream_supported(const Geometry &g)
{
    if (g.ndim != 3 || g.shape != STENCIL_BOX || g.radius != 1)
        return false;
    const int vec = (g.dtype == STENCIL_F32) ? 4 : 2;
    if (lanes_per_row(g, vec) == 0)
        return false;
    // in-plane byte offsets must stay below the out-of-range marker; block counts fit int
    return g.ny * g.nx * int64_t(g.elt) < (int64_t(1) << 30) &&
           g.batch * (g.nx / vec) * g.ny < (int64_t(1) << 30);
}

hipError_t launch_box_stream(const Geometry &g, const void *src, void *dst, const void *field,
                             const void *w, hipStream_t stream)
{
    // 4 rows per lane (tile 1) or 8 (tile 2); the default depends on the coefficient
    // field (the tile resolver states the measurements)
    const int ty = stream_tile(g, 1) == 2 ? 8 : 4;
    if (g.dtype == STENCIL_F32)
        return ty == 4 ? launch_ty<float, 4>(g, src, dst, field, w, stream)
                       : launch_ty<float, 8>(g, src, dst, field, w, stream);
    return ty == 4 ? launch_ty<double, 4>(g, src, dst, field, w, stream)
                   : launch_ty<double, 8>(g, src, dst, field, w, stream);
}

}  // namespace stencil
