// kernel_box2.hip -- 2D box stencils of radius R <= 4 ((2R+1)^2 points), y-streaming,
// gfx950.
//
// This is the operator of the HIERA case study itself (Sec. "Implementation and Evaluation
// Protocol", paragraph "Case-study protocol": a 2D box stencil of radius 3, i.e. a 7x7
// zero-padded cross-correlation with padding 3 and stride 1, in FP64), with any radius up
// to 4, fp32 or fp64, zero or periodic boundary and batched images with per-channel
// weights.  One launch computes one step.
//
// Mapping (no LDS, no barriers):
//   * a wavefront owns a row segment of 64 lanes x 16 bytes (or 64/lpr whole narrower
//     rows, each streamed over its own rows) and streams down a chunk of rows;
//   * each input row is loaded once (16 bytes per lane, prefetched 2R + 1 rows ahead) and
//     folded into 2R + 1 rotating accumulator rows: input row y contributes to output rows
//     y - R .. y + R, so output row y - R is complete and written after row y;
//   * x neighbours come from the lanes up to HXV to the left and right through chained DPP
//     wave shifts; only the first and last lane of a segment load the HXV 16-byte halo
//     vectors beyond it;
//   * buffer loads with 32-bit offsets: rows outside the grid read zero (zero boundary).
#include "common.hpp"
#include "plan.hpp"

#include <type_traits>


namespace stencil {
namespace {

struct Box2Params {
    int ny, nx;
    long long vol;
    int lpr, segw, segs;   // lanes per row segment, segment width, segments per row
    int rg;                // row groups per wavefront (64 / lpr)
    int yc, nyc;           // rows per chunk, chunks per image (per row group)
    long long batch;
    int channels;
    int nblocks;
};

template <typename T, int R, bool PERIODIC, int STORE_CP>
__global__ __launch_bounds__(256) void stencil_box2_stream_kernel(
    const T *__restrict__ in, T *__restrict__ out, const T *__restrict__ w, Box2Params p)
{
    constexpr int VEC = Vec16<T>::N;
    constexpr int E = sizeof(T);
    constexpr int HXV = (R + VEC - 1) / VEC;   // x reach in vectors
    constexpr int NS = 2 * R + 1;              // accumulator rows
    constexpr int NW = 2 * R + 1;              // taps per axis
    constexpr int NX = (2 * HXV + 1) * VEC;    // extended row length (elements)
    constexpr int PF = NS;                     // input rows in flight per lane
    const int lane = threadIdx.x & 63;
    // the wavefront index is uniform by construction; saying so keeps everything derived
    // from it (image, segment, weight pointer, buffer resources) in scalar registers
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

    // work item of this wavefront: (image, segment, chunk); row group rg of the wave takes
    // chunk * rg + its own index, so that narrow rows still use all 64 lanes
    const long long tw = (long long)xcd_logical_block(blockIdx.x, p.nblocks) * 4 + wave;
    const int units = p.segs * p.nyc;  // wavefront work items per image
    const long long b = tw / units;
    if (b >= p.batch)
        return;  // whole wavefront leaves; the kernel has no barriers
    const int t = int(tw - b * units);
    const int seg = t % p.segs;
    const int ch = t / p.segs;  // chunk index of the wavefront (row groups split it)
    const int lx = lane % p.lpr, rgi = lane / p.lpr;
    const int x = seg * p.segw + lx * VEC;
    const int cidx = ch * p.rg + rgi;      // chunk of this row group
    const int y0 = cidx * p.yc;
    // output rows of this row group (0: idle); every row group of the wavefront runs the
    // same number of iterations (p.yc + 2R) so the lane shifts always see active lanes,
    // and stores beyond n are dropped
    const int n = max(0, min(p.yc, p.ny - y0));
    const T *src = in + b * p.vol;
    T *dst = out + b * p.vol;
    const unsigned img_bytes = unsigned(p.vol * E);
    const auto rin = make_rsrc(src, img_bytes);
    const auto rout = make_rsrc(dst, img_bytes);
    const T *wb = w + (b % p.channels) * (NW * NW);

    // halo vectors: the first lane of a segment holds the HXV vectors left of it, the last
    // lane the HXV vectors right of it (a segment has at least two lanes)
    const bool first = lx == 0, last = lx == p.lpr - 1;
    int hx[HXV];
    bool hok[HXV];
#pragma unroll
    for (int k = 0; k < HXV; ++k) {
        int xx = first ? seg * p.segw - (k + 1) * VEC : seg * p.segw + p.segw + k * VEC;
        bool ok = (first || last) && xx >= 0 && xx < p.nx;
        if (PERIODIC) {
            xx = wrap_index(xx, p.nx);
            ok = first || last;
        }
        hx[k] = xx;
        hok[k] = ok;
    }
    // byte offsets of row y: own vector and halo vectors (out of range: reads zero)
    auto row_off = [&](int y, int &own, int (&ho)[HXV]) {
        bool ok = y >= 0 && y < p.ny;
        if (PERIODIC) {
            y = wrap_index(y, p.ny);
            ok = true;
        }
        own = ok ? (y * p.nx + x) * E : kOutOfRange;
#pragma unroll
        for (int k = 0; k < HXV; ++k)
            ho[k] = (ok && hok[k]) ? (y * p.nx + hx[k]) * E : kOutOfRange;
    };

    // rolling queue of PF input rows (row k of the chunk's input is slot k mod PF); the
    // halo vectors (used by two lanes of the segment) are read one row ahead
    Vec16<T> qv[PF], hcur[HXV], hnxt[HXV];
    const int nin = p.yc + 2 * R;  // input rows y0 - R .. y0 + yc - 1 + R
#pragma unroll
    for (int s = 0; s < PF; ++s) {
        int own, ho[HXV];
        row_off(y0 - R + s, own, ho);
        qv[s] = bload16<T>(rin, s < nin ? own : kOutOfRange);
        if (s == 0) {
#pragma unroll
            for (int k = 0; k < HXV; ++k)
                hnxt[k] = bload16<T>(rin, ho[k]);
        }
    }

    T acc[NS][VEC];
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            acc[s][e] = T(0);

    // Fold input row k (y = y0 - R + k).  Offset (a, c) in weight order is (oy, ox) =
    // (a - R, c - R); the input point feeds output row q = k - a (relative to y0), slot
    // q mod NS.  Rows q outside [0, yc) are skipped (uniform across the wavefront).
    auto fold = [&](int k, int pslot, auto slot_of_q) {
        const Vec16<T> own = qv[pslot];
#pragma unroll
        for (int j = 0; j < HXV; ++j)
            hcur[j] = hnxt[j];
        {
            int o1, h1[HXV];
            row_off(y0 - R + k + 1, o1, h1);
#pragma unroll
            for (int j = 0; j < HXV; ++j)
                hnxt[j] = bload16<T>(rin, k + 1 < nin ? h1[j] : kOutOfRange);
        }
        // extended row: vectors of lanes -HXV .. +HXV (halo at the segment's ends)
        Vec16<T> lft[HXV], rgt[HXV];
#pragma unroll
        for (int j = 0; j < HXV; ++j) {
            const Vec16<T> &sl = j == 0 ? own : lft[j - 1];
            const Vec16<T> &sr = j == 0 ? own : rgt[j - 1];
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                const T l = from_left_lane(sl.e[e], hcur[j].e[e]);
                const T r = from_right_lane(sr.e[e], hcur[j].e[e]);
                lft[j].e[e] = first ? hcur[j].e[e] : l;
                rgt[j].e[e] = last ? hcur[j].e[e] : r;
            }
        }
        T ext[NX];
#pragma unroll
        for (int j = 0; j < HXV; ++j)
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                ext[(HXV - 1 - j) * VEC + e] = lft[j].e[e];
                ext[(HXV + 1 + j) * VEC + e] = rgt[j].e[e];
            }
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            ext[HXV * VEC + e] = own.e[e];
        // refill the slot with input row k + PF
        {
            int o2, h2[HXV];
            row_off(y0 - R + k + PF, o2, h2);
            qv[pslot] = bload16<T>(rin, k + PF < nin ? o2 : kOutOfRange);
        }
#pragma unroll
        for (int a = 0; a < NW; ++a) {
            const int q = k - a;
            if (q < 0 || q >= p.yc)
                continue;
            const int s = slot_of_q(a);
#pragma unroll
            for (int c = 0; c < NW; ++c) {
                const T wv = wb[a * NW + c];
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    acc[s][e] = fma(wv, ext[HXV * VEC + e + c - R], acc[s][e]);
            }
        }
        // output row k - 2R is complete (rows before the chunk never received a
        // contribution, so the slot is cleared whatever the row)
        const int qd = k - 2 * R;
        {
            const int sd = slot_of_q(2 * R);
            Vec16<T> v;
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                v.e[e] = acc[sd][e];
                acc[sd][e] = T(0);
            }
            bstore16<T, STORE_CP>(
                rout, (qd >= 0 && qd < n) ? ((y0 + qd) * p.nx + x) * E : kOutOfRange, v);
        }
    };

    // unrolled NS times (PF = NS) so that queue and accumulator slots are static; whole
    // groups in the loop, the remainder after it (an early exit inside the loop body would
    // merge into the loop head and make its waits conservative)
    int k0 = 0;
    for (; k0 + NS <= nin; k0 += NS) {
#pragma unroll
        for (int j = 0; j < NS; ++j)
            fold(k0 + j, j, [j](int a) { return ((j - a) % NS + NS) % NS; });
    }
#pragma unroll
    for (int j = 0; j < NS - 1; ++j)
        if (k0 + j < nin)
            fold(k0 + j, j, [j](int a) { return ((j - a) % NS + NS) % NS; });
}

// Two steps of the 2D box in one pass.  A wavefront's 64 lanes cover a virtual x range
// that starts HXV vectors left of its output columns and ends HXV vectors right of them:
// stage 1 computes u1 on all 64 lanes (the first and last lanes read the u0 halo beyond the
// range), stage 2 folds each completed u1 row into its own accumulators with the lane
// shifts, and only the inner 64 - 2 HXV lanes, whose u1 neighbours are all inside the
// wavefront, are written.  Consecutive wavefronts overlap by 2 HXV lanes.  Under the zero
// boundary u1 is zero outside the grid, exactly as if it had been written and re-read.
// Input row k feeds u1 row k - a (both relative to the chunk), which feeds u2 row
// (k - 2R) - a; with the input queue, both accumulator sets rotate with period 2R + 1.
// At least three wavefronts per SIMD stated explicitly: with per-row buffer resources the
// kernel needs 117 registers for fp64 radius 3 (121 without the hint), which gives four.
// A four-wave hint makes radius 4 spill to scratch.
template <typename T, int R, bool PERIODIC, int STORE_CP>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3))) void
stencil_box2_tb2_kernel(
    const T *__restrict__ in, T *__restrict__ out, const T *__restrict__ w, Box2Params p)
{
    constexpr int VEC = Vec16<T>::N;
    constexpr int E = sizeof(T);
    constexpr int HXV = (R + VEC - 1) / VEC;
    constexpr int NS = 2 * R + 1;
    constexpr int NW = 2 * R + 1;
    constexpr int NX = (2 * HXV + 1) * VEC;
    constexpr int PF = NS;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

    const long long tw = (long long)xcd_logical_block(blockIdx.x, p.nblocks) * 4 + wave;
    const int units = p.segs * p.nyc;
    const long long b = tw / units;
    if (b >= p.batch)
        return;  // whole wavefront leaves; the kernel has no barriers
    const int t = int(tw - b * units);
    const int seg = t % p.segs;
    const int ch = t / p.segs;
    const int xs = seg * p.segw - HXV * VEC;  // virtual x of lane 0 (p.segw: output width)
    const int x = xs + lane * VEC;
    const bool xin = x >= 0 && x < p.nx;
    const bool out_lane = xin && lane >= HXV && lane < 64 - HXV;
    const int out_off = out_lane ? x * E : kOutOfRange;
    const int y0 = ch * p.yc;
    const int n = max(0, min(p.yc, p.ny - y0));
    const T *src = in + b * p.vol;
    T *dst = out + b * p.vol;
    const T *wb = w + (b % p.channels) * (NW * NW);

    const bool first = lane == 0, last = lane == 63;
    auto wrap_x = [&](int xx, bool &ok) {
        ok = xx >= 0 && xx < p.nx;
        if (PERIODIC) {
            xx = wrap_index(xx, p.nx);
            ok = true;
        }
        return xx;
    };
    bool own_ok;
    const int xo = wrap_x(x, own_ok);
    int hx[HXV];
    bool hok[HXV];
#pragma unroll
    for (int k = 0; k < HXV; ++k) {
        hx[k] = wrap_x(first ? xs - (k + 1) * VEC : xs + 64 * VEC + k * VEC, hok[k]);
        hok[k] = hok[k] && (first || last);
    }
    // Addressing: a buffer resource per row, built from wave-uniform values only (scalar
    // work), and per-lane byte offsets within a row that never change.  A row outside
    // the grid (zero boundary) or past the chunk's input gets zero records, so its loads
    // return zero; an invalid lane offset is past any row.  Against per-lane offsets into
    // one image-wide resource: 145 -> 117 VGPRs and 3% less time per step (10240^2 fp64,
    // radius 3).
    const int own_off = own_ok ? xo * E : kOutOfRange;
    int halo_off[HXV];
#pragma unroll
    for (int k = 0; k < HXV; ++k)
        halo_off[k] = hok[k] ? hx[k] * E : kOutOfRange;
    const unsigned row_bytes = unsigned(p.nx * E);
    // a row outside the grid keeps its address (never dereferenced: zero records), which
    // leaves the address affine in the row index, without a select
    auto row_rsrc = [&](int y, bool live) {
        if (PERIODIC)
            return make_rsrc(src + (long long)wrap_index(y, p.ny) * p.nx, live ? row_bytes : 0u);
        const bool ok = live && unsigned(y) < unsigned(p.ny);  // 0 <= y < ny
        return make_rsrc(src + (long long)y * p.nx, ok ? row_bytes : 0u);
    };

    // input rows y0 - 2R .. y0 + yc - 1 + 2R; u1 rows y0 - R .. y0 + yc - 1 + R
    const int nin = p.yc + 4 * R;
    const int n1 = p.yc + 2 * R;
    Vec16<T> qv[PF], hcur[HXV], hnxt[HXV];
#pragma unroll
    for (int s = 0; s < PF; ++s) {
        const auto rr = row_rsrc(y0 - 2 * R + s, true);
        qv[s] = bload16<T>(rr, own_off);
        if (s == 0) {
#pragma unroll
            for (int k = 0; k < HXV; ++k)
                hnxt[k] = bload16<T>(rr, halo_off[k]);
        }
    }
    T acc1[NS][VEC], acc2[NS][VEC];
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            acc1[s][e] = T(0);
            acc2[s][e] = T(0);
        }

    // the 2 HXV + 1 vectors around this lane: DPP shifts.  A shift hands lane 0 (lane 63)
    // the `fix` vector as its left (right) neighbour -- the u0 halo for stage 1, zero for
    // stage 2 -- and chained shifts pass fix[0] on to lane 1, so no select is needed
    // (removing the selects measured 4.6% faster on 10240^2 fp64, radius 3)
    // (ZERO_EDGE: the edge lanes receive zero, through the shifts' bound control, which
    // saves initialising each shift's destination with the fix value)
    auto extend = [&](const Vec16<T> &own, const Vec16<T>(&fix)[HXV], T(&ext)[NX],
                      auto zero_edge) {
        Vec16<T> lft[HXV], rgt[HXV];
#pragma unroll
        for (int j = 0; j < HXV; ++j) {
            const Vec16<T> &sl = j == 0 ? own : lft[j - 1];
            const Vec16<T> &sr = j == 0 ? own : rgt[j - 1];
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                if (decltype(zero_edge)::value) {
                    lft[j].e[e] = from_left_lane_or_zero(sl.e[e]);
                    rgt[j].e[e] = from_right_lane_or_zero(sr.e[e]);
                } else {
                    lft[j].e[e] = from_left_lane(sl.e[e], fix[j].e[e]);
                    rgt[j].e[e] = from_right_lane(sr.e[e], fix[j].e[e]);
                }
            }
        }
#pragma unroll
        for (int j = 0; j < HXV; ++j)
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                ext[(HXV - 1 - j) * VEC + e] = lft[j].e[e];
                ext[(HXV + 1 + j) * VEC + e] = rgt[j].e[e];
            }
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            ext[HXV * VEC + e] = own.e[e];
    };

    // stage 2: fold completed u1 row r1 (in accumulator slot (j + 1) mod NS) into the u2
    // accumulators; arithmetic only, so the caller's branch around it holds no memory access
    auto fold2 = [&](int j, int r1) {
        const int s1 = (j + 1) % NS;
        Vec16<T> u1;
        const int y1 = y0 - R + r1;
        const bool keep = PERIODIC || (xin && y1 >= 0 && y1 < p.ny);
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            u1.e[e] = keep ? acc1[s1][e] : T(0);
            acc1[s1][e] = T(0);
        }
        T ext2[NX];
        Vec16<T> nofix[HXV];
#pragma unroll
        for (int i = 0; i < HXV; ++i)
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                nofix[i].e[e] = T(0);
        extend(u1, nofix, ext2, std::true_type{});
#pragma unroll
        for (int a = 0; a < NW; ++a) {
            const int r2 = r1 - a;
            if (r2 < 0 || r2 >= p.yc)
                continue;
            const int s = ((j + 1 - a) % NS + NS) % NS;
#pragma unroll
            for (int c = 0; c < NW; ++c) {
                const T wv = wb[a * NW + c];
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    acc2[s][e] = fma(wv, ext2[HXV * VEC + e + c - R], acc2[s][e]);
            }
        }
    };

    auto step = [&](int k, int j) {
        // ---- stage 1: input row k -------------------------------------------------
        const Vec16<T> own = qv[j];
#pragma unroll
        for (int i = 0; i < HXV; ++i)
            hcur[i] = hnxt[i];
        {
            const auto rr = row_rsrc(y0 - 2 * R + k + 1, k + 1 < nin);
#pragma unroll
            for (int i = 0; i < HXV; ++i)
                hnxt[i] = bload16<T>(rr, halo_off[i]);
        }
        T ext[NX];
        extend(own, hcur, ext, std::false_type{});
        qv[j] = bload16<T>(row_rsrc(y0 - 2 * R + k + PF, k + PF < nin), own_off);
#pragma unroll
        for (int a = 0; a < NW; ++a) {
            const int r1 = k - a;
            if (r1 < 0 || r1 >= n1)
                continue;
            const int s = ((j - a) % NS + NS) % NS;
#pragma unroll
            for (int c = 0; c < NW; ++c) {
                const T wv = wb[a * NW + c];
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    acc1[s][e] = fma(wv, ext[HXV * VEC + e + c - R], acc1[s][e]);
            }
        }
        // ---- u1 row k - 2R is complete: fold it into stage 2 ---------------------------
        const int r1 = k - 2 * R;
        if (r1 >= 0 && r1 < n1)
            fold2(j, r1);
        // ---- u2 row k - 4R is complete (rows before the chunk never received a
        // contribution, so the slot is cleared whatever the row) --------------------------
        const int r2 = k - 4 * R;
        {
            const int s2 = (j + 2) % NS;
            Vec16<T> v;
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                v.e[e] = acc2[s2][e];
                acc2[s2][e] = T(0);
            }
            const bool live = r2 >= 0 && r2 < n;
            bstore16<T, STORE_CP>(
                make_rsrc(dst + (long long)(y0 + r2) * p.nx, live ? row_bytes : 0u),
                out_off, v);
        }
    };

    // whole groups in the loop, the remainder after it (as in the one-step kernel)
    int k0 = 0;
    for (; k0 + NS <= nin; k0 += NS) {
#pragma unroll
        for (int j = 0; j < NS; ++j)
            step(k0 + j, j);
    }
#pragma unroll
    for (int j = 0; j < NS - 1; ++j)
        if (k0 + j < nin)
            step(k0 + j, j);
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

// Wavefront count of a launch: at most `target` waves (whole rounds of the waves the GPU
// holds at once, scaled by the plan's grid_scale), in whole chunks per image.  A partly
// filled last round leaves the GPU idle for most of its length: on 10240^2 fp64, radius 3,
// 4128 waves against 3072 resident ran 1.34 rounds.
inline long long whole_chunks(long long target, long long per_image, long long max_chunks)
{
    long long nchunks = target / per_image;
    if (nchunks > max_chunks)
        nchunks = max_chunks;
    return nchunks < 1 ? 1 : nchunks;
}

template <typename T, int R>
Box2Params make_params(const Geometry &g, int resident_waves)
{
    constexpr int VEC = Vec16<T>::N;
    Box2Params p{};
    p.ny = int(g.ny);
    p.nx = int(g.nx);
    p.vol = g.vol;
    p.lpr = lanes_per_row(g, VEC);
    p.segw = p.lpr * VEC;
    p.segs = p.nx / p.segw;
    p.rg = 64 / p.lpr;
    p.batch = g.batch;
    p.channels = g.channels;
    // one round of wavefronts; chunks of at least 16 radii of rows so the 2R-row overlap
    // between chunks stays small
    const long long target = scaled_target(resident_waves, g.grid_scale);
    const long long per_image = g.batch * p.segs;
    const long long min_len = 16 * R;
    const long long nchunks =
        whole_chunks(target * p.rg, per_image, (p.ny + min_len - 1) / min_len);
    // chunks are taken rg at a time by a wavefront
    long long total = ((nchunks + p.rg - 1) / p.rg) * p.rg;
    p.yc = int((p.ny + total - 1) / total);
    p.nyc = int(((p.ny + p.yc - 1) / p.yc + p.rg - 1) / p.rg);
    const long long waves = g.batch * p.segs * p.nyc;
    p.nblocks = int((waves + 3) / 4);
    return p;
}

template <typename T, int R>
Box2Params make_tb2_params(const Geometry &g, int resident_waves)
{
    constexpr int VEC = Vec16<T>::N;
    constexpr int HXV = (R + VEC - 1) / VEC;
    Box2Params p{};
    p.ny = int(g.ny);
    p.nx = int(g.nx);
    p.vol = g.vol;
    p.lpr = 64;
    p.segw = (64 - 2 * HXV) * VEC;  // output columns per wavefront
    p.segs = int((g.nx + p.segw - 1) / p.segw);
    p.rg = 1;
    p.batch = g.batch;
    p.channels = g.channels;
    // two rounds of whole chunks: on 10240^2 fp64, radius 3, 0.2747 ms per step for one
    // round, 0.2695 for two, 0.2691 for three, 0.272 for six or eight (the later rounds
    // even out the chunk tails; below 32R rows the 4R-row start-up of each chunk costs
    // more than that)
    const long long target = scaled_target(2LL * resident_waves, g.grid_scale);
    const long long per_image = g.batch * p.segs;
    const long long nchunks =  // >= 32R rows per chunk
        whole_chunks(target, per_image, (p.ny + 32 * R - 1) / (32 * R));
    p.yc = int((p.ny + nchunks - 1) / nchunks);
    p.nyc = (p.ny + p.yc - 1) / p.yc;
    const long long waves = g.batch * p.segs * p.nyc;
    p.nblocks = int((waves + 3) / 4);
    return p;
}

template <typename T, int R, int CP>
hipError_t launch_tb2_cp(const Geometry &g, const void *src, void *dst, const void *w,
                         hipStream_t stream)
{
    const T *s = static_cast<const T *>(src);
    T *d = static_cast<T *>(dst);
    const T *wt = static_cast<const T *>(w);
    if (g.boundary == STENCIL_PERIODIC) {
        const auto k = stencil_box2_tb2_kernel<T, R, true, CP>;
        static const int resident = 4 * resident_blocks(k, 256);
        const Box2Params p = make_tb2_params<T, R>(g, resident);
        k<<<dim3(p.nblocks), dim3(256), 0, stream>>>(s, d, wt, p);
    } else {
        const auto k = stencil_box2_tb2_kernel<T, R, false, CP>;
        static const int resident = 4 * resident_blocks(k, 256);
        const Box2Params p = make_tb2_params<T, R>(g, resident);
        k<<<dim3(p.nblocks), dim3(256), 0, stream>>>(s, d, wt, p);
    }
    return hipGetLastError();
}

template <typename T, int R, int CP>
hipError_t launch_cp(const Geometry &g, const void *src, void *dst, const void *w,
                     hipStream_t stream)
{
    const T *s = static_cast<const T *>(src);
    T *d = static_cast<T *>(dst);
    const T *wt = static_cast<const T *>(w);
    if (g.boundary == STENCIL_PERIODIC) {
        const auto k = stencil_box2_stream_kernel<T, R, true, CP>;
        static const int resident = 4 * resident_blocks(k, 256);
        const Box2Params p = make_params<T, R>(g, resident);
        k<<<dim3(p.nblocks), dim3(256), 0, stream>>>(s, d, wt, p);
    } else {
        const auto k = stencil_box2_stream_kernel<T, R, false, CP>;
        static const int resident = 4 * resident_blocks(k, 256);
        const Box2Params p = make_params<T, R>(g, resident);
        k<<<dim3(p.nblocks), dim3(256), 0, stream>>>(s, d, wt, p);
    }
    return hipGetLastError();
}

template <typename T, int R>
hipError_t launch_r(const Geometry &g, const void *src, void *dst, const void *w, int depth,
                    hipStream_t stream)
{
    const bool nt = streaming_stores(g);
    if (depth == 2)
        return nt ? launch_tb2_cp<T, R, kNonTemporal>(g, src, dst, w, stream)
                  : launch_tb2_cp<T, R, 0>(g, src, dst, w, stream);
    return nt ? launch_cp<T, R, kNonTemporal>(g, src, dst, w, stream)
              : launch_cp<T, R, 0>(g, src, dst, w, stream);
}

template <typename T>
hipError_t launch_t(const Geometry &g, const void *src, void *dst, const void *w, int depth,
                    hipStream_t stream)
{
    switch (g.radius) {
    case 1: return launch_r<T, 1>(g, src, dst, w, depth, stream);
    case 2: return launch_r<T, 2>(g, src, dst, w, depth, stream);
    case 3: return launch_r<T, 3>(g, src, dst, w, depth, stream);
    case 4: return launch_r<T, 4>(g, src, dst, w, depth, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace

bool box2_stream_supported(const Geometry &g)
{
    if (g.ndim != 2 || g.shape != STENCIL_BOX || g.radius < 1 || g.radius > 4 || g.field)
        return false;
    const int vec = (g.dtype == STENCIL_F32) ? 4 : 2;
    if (lanes_per_row(g, vec) == 0)
        return false;
    // 32-bit byte offsets within one image; block count fits int
    return g.vol * int64_t(g.elt) < (int64_t(1) << 30) &&
           g.batch * (g.nx / vec) < (int64_t(1) << 30);
}

bool box2_tb2_supported(const Geometry &g)
{
    // the one-step kernel must also run the shape: odd step counts end with a single step
    return box2_stream_supported(g);
}

hipError_t launch_box2_stream(const Geometry &g, const void *src, void *dst, const void *w,
                              int depth, hipStream_t stream)
{
    if (g.dtype == STENCIL_F32)
        return launch_t<float>(g, src, dst, w, depth, stream);
    return launch_t<double>(g, src, dst, w, depth, stream);
}

}  // namespace stencil
